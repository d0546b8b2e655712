// The decode GEMV kernel template (k_gemv).
#pragma once

#include "dev_common.cuh"

namespace {

// ------------------------------------------------------------ decode GEMV
// Lanes are split into segments of LPR lanes; a segment owns one vocabulary
// row at a time and walks along d in 16-byte chunks (32 codes), LPR chunks
// per iteration, so each segment load is LPR * 16 contiguous bytes.  A wave
// step covers kRowsPerStep rows per segment (WR rows in all); steps are dealt
// out grid-stride over a persistent grid of every resident wave.  x, the chunk
// biases and t sit in LDS.  Step bases are wave-uniform (scalar registers);
// per-lane offsets are 32-bit and computed once per step.  Rows past V (the
// last step only) are clamped to row V-1 for loading and never stored.
struct GemvArgs {
  const uint8_t* codes;
  const uint16_t* rs;
  const int8_t* cu;
  const uint16_t* su;
  const int8_t* ca;
  const uint16_t* sa;
  const uint16_t* x;
  int64_t ldx;
  const uint16_t* rrs;  // fp16 row scales of 8-bit residual scale codes (else unused)
  Stage1Ops s1;    // t of the pass's tokens, computed in the launch
  int n_prod_blocks;  // leading workgroups that compute t
  int64_t tok0;    // first token of this pass
  int64_t V;
  int d, g, rc, rr;
  int gshift;      // log2(g / 32) when g is a power of two, else -1
  int fast;        // the pipelined path applies: expansion codes as dwords (see
                   // ExpOps), d/g even and at most 2 LPR groups per row
  int64_t cu_stride, ca_stride, su_stride, sa_stride;  // 0 for an absent factor
                   // (cu_stride: bytes per row of U_c, int8 codes or ARCHEAD_I5 words)
  int u5;          // U_c codes are ARCHEAD_I5 words
  int64_t cu_bytes, ca_bytes;  // bytes of the U_c / A_w code buffers (V rows)
  int nit;         // iterations along d: (d / 32) / LPR
  int64_t nsteps;  // ceil(V / rows per wave step)
  void* out;
  int64_t ldo;
  int out_bf16;
  // fused CE
  const void* tgt;
  int tgt64;
  float2* part;    // [M, n_part]
  int* part_idx;   // [M, n_part] argmax partials, or null
  int64_t n_part;
  float* tgt_logit;  // [M]
  // fused top-k (single-token variants): per workgroup the k best
  // (logit, index) pairs of the token, [n_part][k]
  float* tk_val;
  int* tk_idx;
  int tk_k;
};

// Sum RB per-lane values over the LPR lanes of each segment.  The first
// log2(RB) butterfly stages halve the number of values per lane (a lane keeps
// one half, its partner the other), so 8 rows cost 7 exchanges + 3 instead of
// 8 * log2(LPR).  Afterwards every lane holds the total of the row given by
// row_of_lane.  Written with compile-time indices throughout so the values
// stay in registers (a runtime index would turn the selects into an indexed
// array access).
__device__ __forceinline__ void xchg_add(float& lo, float hi_v, bool hi, int off) {
  const float send = hi ? lo : hi_v;
  const float keep = hi ? hi_v : lo;
  lo = keep + __shfl_xor(send, off, 64);
}

template <int J, int H, int RB>
__device__ __forceinline__ void xchg_range(float (&v)[RB], bool hi, int off) {
  if constexpr (J < H) {
    xchg_add(v[J], v[J + H], hi, off);
    xchg_range<J + 1, H, RB>(v, hi, off);
  }
}

template <int OFF, int N, int RB>
__device__ __forceinline__ void reduce_stage(float (&v)[RB], int lane) {
  if constexpr (OFF >= 1) {
    if constexpr (N > 1) {
      xchg_range<0, N / 2, RB>(v, (lane & OFF) != 0, OFF);
      reduce_stage<OFF / 2, N / 2, RB>(v, lane);
    } else {
      v[0] += __shfl_xor(v[0], OFF, 64);
      reduce_stage<OFF / 2, 1, RB>(v, lane);
    }
  }
}

template <int LPR, int RB>
__device__ __forceinline__ float seg_reduce_rows(float (&v)[RB], int lane) {
  static_assert(LPR >= RB, "needs at least one lane per row");
  reduce_stage<LPR / 2, RB, RB>(v, lane);
  return v[0];
}

// A pointer every lane of the wave holds, moved to scalar registers so
// loads can use the scalar-base + 32-bit-offset addressing form.
#define ARCHEAD_GLOBAL __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ const ARCHEAD_GLOBAL T* wave_uniform(const T* p) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(u));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(u >> 32));
  return reinterpret_cast<const ARCHEAD_GLOBAL T*>((uint64_t(hi) << 32) | lo);
}

// Row (0..RB-1) whose total seg_reduce_rows leaves in this lane.
template <int LPR, int RB>
__device__ __forceinline__ int row_of_lane(int lane) {
  int r = 0, n = RB;
#pragma unroll
  for (int off = LPR / 2; off > 0 && n > 1; off >>= 1) {
    n /= 2;
    if (lane & off) r += n;
  }
  return r;
}

// Rank-r expansion operands of a step's rows, loaded with the step's first
// chunk of codes.  The (r_c + r_r) / 4 dwords of a row -- U_c codes first,
// then A_w codes -- are dealt to the lanes of its segment, KD per lane: lane
// sl holds dwords q = sl + kd * LPR (4 codes each) and the matching row
// scale (s_U for a U_c dword, s_A for an A_w dword).  Since t is laid out as
// [t_c | t_w], dword q pairs with t[4q .. 4q + 3] in both cases.  Used when
// r_c and r_r are multiples of 4 and (r_c + r_r) / 4 <= KD * LPR.
template <int RB, int KD>
struct ExpOps {
  uint32_t c[RB][KD];   // four int8 codes (general reads: the raw words, decoded when applied)
  RawCodes4 raw[RB][KD];
  uint16_t rsc[RB];     // fp16 row scale of 8-bit residual scale codes (unused otherwise)
  uint16_t s[RB][KD];   // fp16 bit pattern of the row scale (kept 16-bit: no extension op right after the load)
};

template <int LPR>
struct ExpLanes {
  static constexpr int KD = LPR >= 64 ? 1 : 2;
};

// acc += scale * (codes . t) over the lane's dwords of each row.  t is held
// per token as [U_c part | A_w part], each part padded with zeros to a
// multiple of 4 dimensions: R4 dwords of codes per row, Rp = 4 R4 values.
// General reads (GEN > 0): the codes come as raw words; row v0 + rb SEG's
// int8 codes start at byte offset (v cu_st) & 3 (U_c) or (v ca_st) & 3 (A_w)
// of their aligned word (k0 is a multiple of 4).
template <int TOK, int RB, int KD, int LPR, int GEN = 0>
__device__ __forceinline__ void apply_expansion(float (&acc)[RB][TOK], const ExpOps<RB, KD>& e,
                                                const float* st, int R4, int sl, int rc4 = 0,
                                                int64_t v0 = 0, int seg_rows = 0,
                                                int64_t cu_st = 0, int64_t ca_st = 0) {
  const int Rp = 4 * R4;
#pragma unroll
  for (int kd = 0; kd < KD; ++kd) {
    const int q = sl + kd * LPR;
    const bool valid = q < R4;
    const int qq = valid ? q : 0;
#pragma unroll
    for (int tt = 0; tt < TOK; ++tt) {
      const float4 t4 = *reinterpret_cast<const float4*>(st + tt * Rp + 4 * qq);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        uint32_t u;
        if constexpr (GEN > 0) {
          const uint32_t v = uint32_t(v0 + int64_t(rb) * seg_rows);
          const bool isu = qq < rc4;
          const uint32_t sh = (v * uint32_t(isu ? cu_st : ca_st)) & 3u;
          u = isu ? fcodes4_decode<GEN == 2>(e.raw[rb][kd], 4 * qq, sh)
                  : fcodes4_decode<false>(e.raw[rb][kd], 4 * (qq - rc4), sh);
        } else {
          u = e.c[rb][kd];
        }
        float du = float(int8_t(u)) * t4.x;
        du = fmaf(float(int8_t(u >> 8)), t4.y, du);
        du = fmaf(float(int8_t(u >> 16)), t4.z, du);
        du = fmaf(float(int8_t(u >> 24)), t4.w, du);
        // a lane without a dword read t4 from t[0..3], or with r_c + r_r = 0
        // from LDS past t (stale bits, possibly NaN): drop du, not just its scale
        du = valid ? du : 0.f;
        const float sc = valid ? f16_to_f32(uint16_t(e.s[rb][kd])) : 0.f;
        acc[rb][tt] = fmaf(sc, du, acc[rb][tt]);
      }
    }
  }
}

// One d-iteration of a step: RB rows x one 16-byte chunk per lane.
template <int TOK, int RB, bool SC8>
__device__ __forceinline__ void gemv_chunk(float (&acc)[RB][TOK], const uint4 (&q)[RB],
                                           const uint32_t (&sc)[RB], const uint16_t* sx,
                                           const float* sxb, int d, int C, int c,
                                           uint32_t kMask, uint32_t kMagic) {
  uint32_t xw[TOK][16];
  float xb[TOK];
#pragma unroll
  for (int tt = 0; tt < TOK; ++tt) {
    // x is held in LDS as [token][part j][chunk c] of 16-byte units, so the
    // lanes of a wave (consecutive chunks) read consecutive 16-byte units
    const uint4* px = reinterpret_cast<const uint4*>(sx) + tt * 4 * C + c;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint4 u = px[j * C];
      xw[tt][4 * j] = u.x; xw[tt][4 * j + 1] = u.y;
      xw[tt][4 * j + 2] = u.z; xw[tt][4 * j + 3] = u.w;
    }
    xb[tt] = sxb[tt * C + c];
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    // the group scale: fp16, or an 8-bit code (the row scale is applied at
    // the step's end)
    const float s = SC8 ? float(sc[rb] & 0xffu) : f16_to_f32(uint16_t(sc[rb]));
    const uint32_t w4[4] = {q[rb].x, q[rb].y, q[rb].z, q[rb].w};
    uint32_t pr[16];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      pr[4 * w + 0] = int4_pair<0>(w4[w], kMask, kMagic);
      pr[4 * w + 1] = int4_pair<1>(w4[w], kMask, kMagic);
      pr[4 * w + 2] = int4_pair<2>(w4[w], kMask, kMagic);
      pr[4 * w + 3] = int4_pair<3>(w4[w], kMask, kMagic);
    }
#pragma unroll
    for (int tt = 0; tt < TOK; ++tt) {
      float dsum = xb[tt];
#pragma unroll
      for (int j = 0; j < 16; ++j) dsum = dot2_bf16(pr[j], xw[tt][j], dsum);
      acc[rb][tt] = fmaf(s, dsum, acc[rb][tt]);
    }
  }
}

// End of a step: add the rank-r expansions of the lane's rows, reduce over
// the segment and store the logits (or fold them into the softmax state).
// Row rb of the lane is row0 + min(seg + rb * SEG, lim).
template <int TOK, int LPR, int RB, bool CE, bool EXPAND, bool TK>
__device__ __forceinline__ void gemv_epilogue(float (&acc)[RB][TOK], const GemvArgs& a,
                                              int64_t row0, uint32_t lim, int seg, int sl,
                                              int lane, int my_row, bool writer,
                                              const float* st, CeState<TOK>& ce) {
  constexpr int SEG = 64 / LPR;
  const int rcp = 4 * ((a.rc + 3) / 4);           // padded U_c part of t
  const int Rp = rcp + 4 * ((a.rr + 3) / 4);
#pragma unroll
  for (int rb = 0; rb < RB && EXPAND; ++rb) {
    uint32_t r = uint32_t(seg + rb * SEG);
    r = r < lim ? r : lim;
    const int64_t v = row0 + r;
    if (a.rc) {
      const float su = f16_to_f32(a.su[v]);
      const uint8_t* urow = reinterpret_cast<const uint8_t*>(a.cu) + v * a.cu_stride;
      for (int k = sl; k < a.rc; k += LPR) {
        const float u = su * float(fcode1(urow, k, a.u5 != 0));
#pragma unroll
        for (int tt = 0; tt < TOK; ++tt) acc[rb][tt] = fmaf(u, st[tt * Rp + k], acc[rb][tt]);
      }
    }
    if (a.rr) {
      const float sa = f16_to_f32(a.sa[v]);
      for (int k = sl; k < a.rr; k += LPR) {
        const float u = sa * float(a.ca[v * a.rr + k]);
#pragma unroll
        for (int tt = 0; tt < TOK; ++tt)
          acc[rb][tt] = fmaf(u, st[tt * Rp + rcp + k], acc[rb][tt]);
      }
    }
  }
  const int64_t v = row0 + seg + int64_t(my_row) * SEG;   // row this lane reports
  const bool store = writer && v < a.V;
#pragma unroll
  for (int tt = 0; tt < TOK; ++tt) {
    float col[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) col[rb] = acc[rb][tt];
    const float l = seg_reduce_rows<LPR, RB>(col, lane);
    if constexpr (TK) {
      tk_offer(ce.tv[tt], ce.ti[tt], ce.bv[tt], ce.bi[tt], l, int(v), store, lane, a.tk_k);
    } else if (store) {
      if constexpr (!CE) {
        const int64_t o = (a.tok0 + tt) * a.ldo + v;
        if (a.out_bf16)
          reinterpret_cast<uint16_t*>(a.out)[o] = f32_to_bf16_rne(l);
        else
          reinterpret_cast<float*>(a.out)[o] = l;
      } else {
        // a lane's rows come in increasing order: the first of equal
        // maxima is the smallest index
        if (l > ce.mx[tt]) {
          ce.se[tt] = ce.se[tt] * fast_exp(ce.mx[tt] - l) + 1.f;
          ce.mx[tt] = l;
          ce.am[tt] = int(v);
        } else {
          ce.se[tt] += fast_exp(l - ce.mx[tt]);
        }
        if (v == ce.y[tt]) a.tgt_logit[a.tok0 + tt] = l;
      }
    }
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int tt = 0; tt < TOK; ++tt) acc[rb][tt] = 0.f;
}

// Waves per SIMD the single-token GEMV is compiled for (register budget
// 512 / waves per lane).
#ifndef ARCHEAD_GEMV_WAVES
#define ARCHEAD_GEMV_WAVES 3
#endif
#ifndef ARCHEAD_GEMV_WAVES_NARROW
#define ARCHEAD_GEMV_WAVES_NARROW 2   // segments narrower than the wave
#endif
// GEN: how the pipelined path reads the rank-r codes: 0 as aligned dwords
// (int8 codes, ranks that are multiples of 4); 1 through fcodes4 (int8 codes,
// any rank); 2 the same with the core-left codes in ARCHEAD_I5 words.
// TK: the single-token top-k variant (no logit store; CE false).
template <int TOK, int LPR, bool CE, bool SC8, int GEN, bool TK = false>
__global__ __launch_bounds__(kBlock)
__attribute__((amdgpu_waves_per_eu(TOK == 1 ? (LPR >= 64 ? ARCHEAD_GEMV_WAVES : ARCHEAD_GEMV_WAVES_NARROW) : 1)))
void k_gemv(GemvArgs a) {
  constexpr int SEG = 64 / LPR;              // rows in flight per wave
  constexpr int RB = LPR < kRowsPerStep ? LPR : kRowsPerStep;
  constexpr int WR = RB * SEG;               // rows per wave step
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ float2 red[kWaves][TOK];
  __shared__ int redi[kWaves][TOK];

  const int d = a.d;
  const int C = d / 32;                      // 16-byte chunks per row
  const int R = a.rc + a.rr;
  const int rcq = (a.rc + 3) / 4, Rq = rcq + (a.rr + 3) / 4;  // dwords of codes per row
  const int Rp = 4 * Rq;                                      // t per token, parts padded
  uint16_t* sx = reinterpret_cast<uint16_t*>(smem);          // [TOK][d]
  float* sxb = reinterpret_cast<float*>(sx + TOK * d);        // [TOK][C]
  const int wid = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  float* st = sxb + TOK * C + wid * TOK * Rp;                 // this wave's t [TOK][Rp]
  // x[tt][i .. i + 7] and x[tt][i], x[tt][i + 1] in the chunked LDS layout
  auto x8 = [&](int tt, int i) {
    return *reinterpret_cast<const u32x4_t*>(
        reinterpret_cast<const uint4*>(sx) + (tt * 4 + ((i >> 3) & 3)) * C + (i >> 5));
  };
  auto x2 = [&](int tt, int i) {
    return *reinterpret_cast<const uint32_t*>(
        reinterpret_cast<const uint8_t*>(reinterpret_cast<const uint4*>(sx) +
                                         (tt * 4 + ((i >> 3) & 3)) * C + (i >> 5)) +
        2 * (i & 7));
  };

  // x into LDS (chunked layout) and the chunk biases -136 * (sum of x over
  // the chunk); every wave of the workgroup calls this once
  auto prologue = [&]() {
    const int x8n = d / 8;  // 16-byte units per token: unit u = chunk u/4, part u%4
    // each thread's units are requested in batches of 8 before any is
    // stored, so the copy costs one memory latency per batch
    const int nx = TOK * x8n;
    for (int i0 = 0; i0 < nx; i0 += 8 * kBlock) {
      uint4 v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int i0j = i0 + j * kBlock + int(threadIdx.x);
        const int i = i0j < nx ? i0j : nx - 1;   // past the end: a valid unit, not stored
        const int tt = i / x8n, u = i - tt * x8n;
        v[j] = *reinterpret_cast<const uint4*>(a.x + (a.tok0 + tt) * a.ldx + u * 8);
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int i = i0 + j * kBlock + int(threadIdx.x);
        const int tt = i / x8n, u = i - tt * x8n;
        if (i < nx) reinterpret_cast<uint4*>(sx)[(tt * 4 + (u & 3)) * C + (u >> 2)] = v[j];
      }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < TOK * C; i += kBlock) {
      const int tt = i / C, c = i - tt * C;
      float s = 0.f;
      for (int j = 0; j < 4; ++j) {
        const uint4 u = reinterpret_cast<const uint4*>(sx)[(tt * 4 + j) * C + c];
        s += bf16_lo(u.x) + bf16_hi(u.x) + bf16_lo(u.y) + bf16_hi(u.y) +
             bf16_lo(u.z) + bf16_hi(u.z) + bf16_lo(u.w) + bf16_hi(u.w);
      }
      sxb[i] = -float(archead::kInt4Bias) * s;
    }
    __syncthreads();
  };

  const int lane = threadIdx.x & 63;
  // stage-1 producers: one rank row per wave, the pass's tokens
  if (int(blockIdx.x) < a.n_prod_blocks) {
    prologue();
    const int k = int(blockIdx.x) * kWaves + wid;
    if (k < R) s1_produce<TOK>(a.s1, k, TOK, a.tok0, x8, lane);
    return;
  }
  // this wave's copy of t, fetched when first needed (end of its first step)
  bool t_ready = R == 0;
  auto fetch_t = [&]() {
    for (int e = lane; e < TOK * Rp; e += 64) {
      const int tt = e / Rp, j = e - tt * Rp;
      // [U_c dims, zeros to 4 rcq | A_w dims, zeros]
      const int k = j < 4 * rcq ? (j < a.rc ? j : -1) : (j - 4 * rcq < a.rr ? a.rc + j - 4 * rcq : -1);
      st[e] = k >= 0 ? s1_value(a.s1, a.tok0, tt, k, x2) : 0.f;
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    t_ready = true;
  };

  const int seg = lane / LPR, sl = lane % LPR;
  // Steps are dealt out grid-stride (wave gw takes steps gw, gw + W, ...), so
  // at any moment the whole grid streams one compact window of the head.
  const int64_t W = int64_t(gridDim.x - a.n_prod_blocks) * kWaves;
  const int64_t gw = int64_t(blockIdx.x - a.n_prod_blocks) * kWaves + wid;
  const uint32_t rowbytes = uint32_t(d) / 2;
  const uint32_t ngrp = uint32_t(d / a.g);
  const int my_row = row_of_lane<LPR, RB>(lane);   // row this lane ends up with
  const bool writer = (sl & (LPR / RB - 1)) == 0;
  // nibble-pair mask and bf16 128.0 bit pattern, held in registers
  const uint32_t kMask = opaque_vgpr(0x000F000Fu);
  const uint32_t kMagic = opaque_vgpr(0x43004300u);

  CeState<TOK> ce;
#pragma unroll
  for (int tt = 0; tt < TOK; ++tt) {
    ce.mx[tt] = -INFINITY;
    ce.se[tt] = 0.f;
    ce.am[tt] = kNoIdx;
    ce.y[tt] = -1;
    ce.tv[tt] = -INFINITY;
    ce.ti[tt] = kNoIdx;
    ce.bv[tt] = -INFINITY;
    ce.bi[tt] = kNoIdx;
    if constexpr (CE)
      if (a.tgt)
        ce.y[tt] = a.tgt64 ? reinterpret_cast<const int64_t*>(a.tgt)[a.tok0 + tt]
                           : int64_t(reinterpret_cast<const int32_t*>(a.tgt)[a.tok0 + tt]);
  }
  float acc[RB][TOK];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int tt = 0; tt < TOK; ++tt) acc[rb][tt] = 0.f;

  // ---- full steps (every row < V): software-pipelined.  Loads run kPD
  // iterations ahead of the arithmetic in a ring of kPD + 1 register
  // buffers, so a wave keeps about kPD iterations of codes in flight while it
  // computes; codes and scales are read through buffer resources whose base
  // and per-row offsets live in scalar registers.
  const int64_t full_steps = a.fast ? a.V / WR : 0;
  {
    constexpr int kPD = ARCHEAD_GEMV_PREFETCH;
    constexpr int NB = kPD + 1;
    const uint32_t voff = uint32_t(seg) * rowbytes + uint32_t(sl) * 16u;
    const uint32_t svoff = uint32_t(seg) * ngrp;
    // every load below is unconditional: absent factors point at a valid
    // buffer with row stride 0 (see gemv_args), lanes without a dword
    // re-read dword 0, and loads past the wave's last iteration re-read that
    // iteration; all of it is masked or unused, so no branch separates a
    // load from its use (a branch would make the wait-count pass drain the
    // loads in flight)
    constexpr int KD = ExpLanes<LPR>::KD;
    const int rc4 = rcq, R4 = Rq;
    constexpr uint32_t ESZ = SC8 ? 1u : 2u;   // bytes per group scale
    auto load = [&](int64_t stp, int itx, uint4 (&q)[RB], uint32_t (&sc)[RB]) {
      const uint64_t cbytes = uint64_t(a.V - stp * WR) * rowbytes;
      const uint64_t sbytes = uint64_t(a.V - stp * WR) * ngrp * ESZ;
      const __amdgpu_buffer_rsrc_t rc_ = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint8_t*>(a.codes + uint64_t(stp) * WR * rowbytes), 0,
          int(cbytes < 0xffffffffull ? cbytes : 0xffffffffull), kBufferWord3);
      const __amdgpu_buffer_rsrc_t rs_ = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint8_t*>(reinterpret_cast<const uint8_t*>(a.rs) + uint64_t(stp) * WR * ngrp * ESZ), 0,
          int(sbytes < 0xffffffffull ? sbytes : 0xffffffffull), kBufferWord3);
      const int itoff = itx * LPR * 16;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(
            rc_, int(voff), int(uint32_t(rb * SEG) * rowbytes) + itoff, kLoadStream);
        q[rb] = make_uint4(v.x, v.y, v.z, v.w);
      }
      // a step's group scales come with its first iteration: lane sl of a
      // segment takes groups 2 sl, 2 sl + 1 (fp16) or 4 sl .. 4 sl + 3 (8-bit
      // codes) of each of its rows (4 bytes); the lanes that need them fetch
      // them with ds_bpermute
      if (itx == 0) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          sc[rb] = __builtin_amdgcn_raw_buffer_load_b32(
              rs_, int(svoff * ESZ + uint32_t(sl) * 4u), int(uint32_t(rb * SEG) * ngrp * ESZ), 0);
      }
    };
    // expansion operands of step stp (one buffer: the next step's operands
    // are requested right after the current step's have been applied)
    // (the strides pass through registers and the pointers are selected
    // after the offsets are applied, so no per-lane select picks between two
    // fields of the argument block, which the compiler would turn into a
    // vector load of the selected field)
    const int64_t cu_st = GEN ? a.cu_stride : opaque_sgpr(a.cu_stride);
    const int64_t ca_st = GEN ? a.ca_stride : opaque_sgpr(a.ca_stride);
    const int64_t su_st = GEN ? a.su_stride : opaque_sgpr(a.su_stride);
    const int64_t sa_st = GEN ? a.sa_stride : opaque_sgpr(a.sa_stride);
    // resources over the factor-code buffers (general reads: aligned dwords
    // that may reach past a row; past the buffer they read zero)
    // (sizes rounded up to whole dwords: the aligned dword holding a
    // buffer's last bytes must be read whole; what it holds past the buffer
    // is in the same dword and pairs with zero t)
    const __amdgpu_buffer_rsrc_t rcu = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int8_t*>(a.cu), 0, int((a.cu_bytes + 3) & ~int64_t(3)), kBufferWord3);
    const __amdgpu_buffer_rsrc_t rca = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int8_t*>(a.ca), 0, int((a.ca_bytes + 3) & ~int64_t(3)), kBufferWord3);
    auto load_exp = [&](int64_t stp, ExpOps<RB, KD>& e) __attribute__((always_inline)) {
      const int64_t v0 = stp * WR + seg;
#pragma unroll
      for (int kd = 0; kd < KD; ++kd) {
        int q = sl + kd * LPR;
        q = q < R4 ? q : 0;
        const bool isu = q < rc4;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const int64_t v = v0 + rb * SEG;
          const uint16_t* sp = isu ? a.su + v * su_st : a.sa + v * sa_st;
          if constexpr (GEN > 0) {
            // the words only: they are joined when the expansion is applied,
            // so the loads stay in flight through the next step
            e.raw[rb][kd] = isu ? fcodes4_fetch<GEN == 2>(rcu, int(v * cu_st), 4 * q)
                                : fcodes4_fetch<false>(rca, int(v * ca_st), 4 * (q - rc4));
          } else {
            const int8_t* cb = isu ? a.cu + 4 * q + v * cu_st : a.ca + 4 * (q - rc4) + v * ca_st;
            e.c[rb][kd] = *reinterpret_cast<const uint32_t*>(cb);
          }
          e.s[rb][kd] = *sp;
        }
      }
      if constexpr (SC8) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) e.rsc[rb] = a.rrs[v0 + rb * SEG];
      }
    };
    uint4 q[NB][RB];
    uint32_t sc[NB][RB];
    uint32_t ssc[RB];   // the current step's scales (groups 2 sl, 2 sl + 1 of each row)
    ExpOps<RB, KD> e;
    const int64_t last_step = gw + ((full_steps - 1 - gw) / W) * W;
    auto advance = [&](int64_t& st, int& itv) {
      if (++itv == a.nit) { itv = 0; st += W; }
    };
    int64_t cstep = gw, lstep = gw;   // compute and load cursors
    int cit = 0, lit = 0;
    // the first loads of the head go out before the prologue, so the memory
    // works while x and the chunk biases are set up
    if (gw < full_steps) {
#pragma unroll
      for (int j = 0; j < kPD; ++j) {
        const bool ok = lstep < full_steps;
        load(ok ? lstep : last_step, ok ? lit : a.nit - 1, q[j], sc[j]);
        advance(lstep, lit);
      }
      load_exp(cstep, e);
    }
    prologue();
    bool done = false;
    auto body = [&](auto J) {
      constexpr int j = decltype(J)::value;
      constexpr int jl = (j + kPD) % NB;
      {
        const bool ok = lstep < full_steps;
        load(ok ? lstep : last_step, ok ? lit : a.nit - 1, q[jl], sc[jl]);
        advance(lstep, lit);
      }
      asm volatile("" ::: "memory");  // keep the loads ahead of the work below
      int64_t nstep = cstep;
      int nit = cit;
      advance(nstep, nit);
      const bool more = nstep < full_steps;
      if (cit == 0) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) ssc[rb] = sc[j][rb];
      }
      // group of this lane's chunk and the segment lane holding its scale
      const uint32_t c = uint32_t(cit * LPR + sl);
      const uint32_t grp = a.gshift >= 0 ? (c >> a.gshift) : (c * 32u) / uint32_t(a.g);
      const int src = 4 * (seg * LPR + int(SC8 ? grp >> 2 : grp >> 1));
      const uint32_t hsh = SC8 ? (grp & 3u) * 8u : (grp & 1u) * 16u;
      uint32_t scv[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        scv[rb] = uint32_t(__builtin_amdgcn_ds_bpermute(src, int(ssc[rb]))) >> hsh;
      gemv_chunk<TOK, RB, SC8>(acc, q[j], scv, sx, sxb, d, C, int(c), kMask, kMagic);
      if (cit == a.nit - 1) {
        // the step's rank-r expansion, then the next step's operands
        if (!t_ready) fetch_t();
        if constexpr (SC8) {   // the residual in units of the row scales
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            const float f = f16_to_f32(e.rsc[rb]);
#pragma unroll
            for (int tt = 0; tt < TOK; ++tt) acc[rb][tt] *= f;
          }
        }
        apply_expansion<TOK, RB, KD, LPR, GEN>(acc, e, st, Rq, sl, rc4, cstep * WR + seg, SEG,
                                               cu_st, ca_st);
        load_exp(more ? nstep : cstep, e);
        gemv_epilogue<TOK, LPR, RB, CE, false, TK>(acc, a, cstep * WR, uint32_t(WR - 1), seg, sl,
                                               lane, my_row, writer, st, ce);
      }
      cstep = nstep;
      cit = nit;
      done = !more;
    };
    // one pass of the loop takes every ring slot once, in order
    auto body_done = [&](auto J) {
      body(J);
      return done;
    };
    if (gw < full_steps)
      while (!unroll_until<0, NB>(body_done)) {
      }
  }

  // ---- steps not taken above: the partial last step (rows past V clamped
  // to V-1, never stored), or every step when the expansion codes cannot be
  // read as dwords; grid-stride like the fast path
  int64_t first = full_steps + ((gw - full_steps % W) % W + W) % W;
  for (int64_t step = first; step < a.nsteps; step += W) {
    const int64_t row0 = step * WR;
    const uint8_t* cbase = a.codes + row0 * rowbytes;
    const uint16_t* sbase = a.rs + row0 * ngrp;
    const int64_t left = a.V - 1 - row0;
    const uint32_t lim = uint32_t(left < WR - 1 ? left : WR - 1);
    for (int it = 0; it < a.nit; ++it) {
      const uint32_t c = uint32_t(it * LPR + sl);
      const uint32_t grp = a.gshift >= 0 ? (c >> a.gshift) : (c * 32u) / uint32_t(a.g);
      uint4 q[RB];
      uint32_t sc[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        uint32_t r = uint32_t(seg + rb * SEG);
        r = r < lim ? r : lim;
        q[rb] = load_stream16(cbase + uint64_t(r) * rowbytes + c * 16u);
        sc[rb] = SC8 ? reinterpret_cast<const uint8_t*>(a.rs)[uint64_t(row0 + r) * ngrp + grp]
                     : sbase[uint64_t(r) * ngrp + grp];
      }
      gemv_chunk<TOK, RB, SC8>(acc, q, sc, sx, sxb, d, C, int(c), kMask, kMagic);
    }
    if (!t_ready) fetch_t();
    if constexpr (SC8) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        uint32_t r = uint32_t(seg + rb * SEG);
        r = r < lim ? r : lim;
        const float f = f16_to_f32(a.rrs[row0 + r]);
#pragma unroll
        for (int tt = 0; tt < TOK; ++tt) acc[rb][tt] *= f;
      }
    }
    gemv_epilogue<TOK, LPR, RB, CE, true, TK>(acc, a, row0, lim, seg, sl, lane, my_row, writer, st,
                                          ce);
  }

  if constexpr (CE) {
    // (max, sum exp) over the workgroup, and the argmax: the smallest index
    // among the lanes (then waves) whose maximum is the overall one
#pragma unroll
    for (int tt = 0; tt < TOK; ++tt) {
      const float own = ce.mx[tt];
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const float om = __shfl_xor(ce.mx[tt], off, 64);
        const float os = __shfl_xor(ce.se[tt], off, 64);
        lse_merge(ce.mx[tt], ce.se[tt], om, os);
      }
      int ai = own == ce.mx[tt] ? ce.am[tt] : kNoIdx;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) ai = min(ai, __shfl_xor(ai, off, 64));
      if (lane == 0) {
        red[wid][tt] = make_float2(ce.mx[tt], ce.se[tt]);
        redi[wid][tt] = ai;
      }
    }
    __syncthreads();
    if (threadIdx.x < TOK) {
      const int tt = threadIdx.x;
      float m = red[0][tt].x, s = red[0][tt].y;
      for (int w = 1; w < kWaves; ++w) lse_merge(m, s, red[w][tt].x, red[w][tt].y);
      const int64_t o = (a.tok0 + tt) * a.n_part + (blockIdx.x - a.n_prod_blocks);
      a.part[o] = make_float2(m, s);
      if (a.part_idx) {
        int ai = kNoIdx;
        for (int w = 0; w < kWaves; ++w)
          if (red[w][tt].x == m) ai = min(ai, redi[w][tt]);
        a.part_idx[o] = ai;
      }
    }
  }
  if constexpr (TK) {
    // the waves' lists merged by rank into this workgroup's partial
    __shared__ float tks_v[kWaves * 64];
    __shared__ int tks_i[kWaves * 64];
    __shared__ float tko_v[kTopKMax];
    __shared__ int tko_i[kTopKMax];
    const int tid = int(threadIdx.x);
#pragma unroll
    for (int tt = 0; tt < TOK; ++tt) {
      tk_rank_merge<kWaves>(ce.tv[tt], ce.ti[tt], tid, a.tk_k, tks_v, tks_i, tko_v, tko_i);
      if (tid < a.tk_k) {
        const int64_t o = ((a.tok0 + tt) * a.n_part + (blockIdx.x - a.n_prod_blocks)) * a.tk_k + tid;
        a.tk_val[o] = tko_v[tid];
        a.tk_idx[o] = tko_i[tid];
      }
      __syncthreads();
    }
  }
}

}  // namespace
