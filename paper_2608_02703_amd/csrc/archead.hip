// ARCHead packed LM-head forward on gfx950: kernels and the device-side C ABI.
//
// logit[m, v] = sum_j s_res[v, j] sum_{i in group j} c[v, i] x[m, i]
//             + s_U[v] sum_k cU[v, k] t_c[m, k] + s_A[v] sum_k cA[v, k] t_w[m, k]
// (ARCHead Section 3.2: Y_hat = H W_d^T + (H B_w^T) A_w^T with the packed
// core W_d = Q5(A_c) Q8(B_c) + Q_SC4(.)).  t_c = x V_c^T and t_w = x B_w^T
// are formed first (stage 1), then one pass over the packed head evaluates
// the INT4 residual and folds the two rank-r expansions into the same
// vocabulary-row epilogue.
//
// INT4 unpack: a 32-bit word q of ARCHEAD_INT4_V1 holds elements 8w..8w+7;
// ((q >> 4k) & 0x000F000F) | 0x43004300 is the bf16 pair (128 + u) for
// elements (8w+2k, 8w+2k+1), i.e. 136 + c exactly.  The dot product with an
// x pair (v_dot2_f32_bf16, fp32 accumulate) therefore yields
// sum (c + 136) x; the accumulator starts at -136 * sum x over the chunk, so
// the group partial is sum c x.  The group scale multiplies that fp32 partial
// (it is never folded into a bf16 weight).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdlib.h>

#include <type_traits>
#include <stdint.h>
#include <string.h>

#include "archead.h"
#include "internal.h"

namespace {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// 16-byte streaming load (read once: non-temporal hint).
__device__ __forceinline__ uint4 load_stream16(const uint8_t* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint4 load_stream16(const __attribute__((address_space(1))) uint8_t* p) {
  const u32x4_t v = __builtin_nontemporal_load(
      reinterpret_cast<const __attribute__((address_space(1))) u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

constexpr int kBlock = 256;          // 4 waves of 64
constexpr int kWaves = kBlock / 64;
#ifndef ARCHEAD_ROWS_PER_STEP
#define ARCHEAD_ROWS_PER_STEP 8
#endif
#ifndef ARCHEAD_GEMV_BLOCKS_PER_CU
#define ARCHEAD_GEMV_BLOCKS_PER_CU 3
#endif
#ifndef ARCHEAD_GEMV_PREFETCH
#define ARCHEAD_GEMV_PREFETCH 1   // GEMV iterations of loads in flight ahead of compute
#endif
constexpr int kRowsPerStep = ARCHEAD_ROWS_PER_STEP;  // rows per lane segment of a GEMV step
constexpr int kGemvBlocksPerCu = ARCHEAD_GEMV_BLOCKS_PER_CU;  // resident GEMV workgroups per CU
constexpr float kLog2e = 1.4426950408889634f;
// Fourth word of a gfx9 buffer resource for raw (untyped) 32-bit accesses.
constexpr int kBufferWord3 = 0x00020000;
// Cache-policy operand of a buffer load: non-temporal (read-once data).
constexpr int kLoadStream = 2;

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}
__device__ __forceinline__ float f16_to_f32(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);
}
__device__ __forceinline__ float bf16_lo(uint32_t p) { return __uint_as_float(p << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t p) { return __uint_as_float(p & 0xffff0000u); }

// (x & m) | o in one VALU op.  The compiler splits it into v_and + v_or when
// both constants are literals (gfx9 VOP3 has no literal operand), so the
// constants are kept in registers and the fused instruction is named here.
__device__ __forceinline__ uint32_t and_or(uint32_t x, uint32_t m, uint32_t o) {
  uint32_t r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "v"(m), "v"(o));
  return r;
}

// Bf16 pair (136 + c) of INT4_V1 elements (8w + 2k, 8w + 2k + 1) of word q.
template <int K>
__device__ __forceinline__ uint32_t int4_pair(uint32_t q, uint32_t mask, uint32_t magic) {
  return and_or(K ? (q >> (4 * K)) : q, mask, magic);
}

// fp32 -> bf16, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return uint16_t((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

__device__ __forceinline__ float fast_exp(float x) {
  return __builtin_amdgcn_exp2f(x * kLog2e);
}

// (max, sum of exp(l - max)) pairs: merge b into a.
__device__ __forceinline__ void lse_merge(float& mx, float& se, float bmx, float bse) {
  float m = fmaxf(mx, bmx);
  if (m == -INFINITY) return;  // both empty
  se = se * fast_exp(mx - m) + bse * fast_exp(bmx - m);
  mx = m;
}

template <int W>
__device__ __forceinline__ float seg_sum(float v) {
#pragma unroll
  for (int off = W / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// ------------------------------------------------------------------ stage 1
// t[m, k] = sum_i (s[k, i/grp] c[k, i]) x[m, i] for the rows k of V_c (k <
// r_c) then of B_w.  One workgroup per (k, block of 8 tokens): the 256
// threads split d in 8-element pieces, every load of the row is issued before
// the arithmetic, and the block sums the 256 partials.  s * c is exact in fp32
// (11 x 8 significant bits).
struct Stage1Args {
  const uint16_t* x;
  int64_t ldx, M, d;
  const int8_t* cv;
  const uint16_t* sv;
  int64_t gv, rc;
  const int8_t* cb;
  const uint16_t* sb;
  int64_t gb, rr;
  float* t;  // [M, rc + rr]
  int64_t mbase;  // first token of this launch
  float* xs;      // [M, d/g] per-group sums of x (MFMA path), or null
  int64_t g;
};

constexpr int kS1Tok = 8;
constexpr int64_t kMaxGridY = 65535;

__global__ __launch_bounds__(kBlock) void k_stage1(Stage1Args a) {
  __shared__ float red[kWaves][kS1Tok];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int64_t R = a.rc + a.rr;
  const int64_t k = blockIdx.x, m0 = a.mbase + int64_t(blockIdx.y) * kS1Tok;
  if (k >= R) {
    // per-group sums xs[m, j] = sum over group j of x[m, i] (bias of the MFMA
    // kernel's offset-binary unpack); one workgroup per (group, token block)
    const int64_t j = k - R, ngrp = a.d / a.g;
    const int ntok = int(a.M - m0 < kS1Tok ? a.M - m0 : kS1Tok);
    float acc[kS1Tok];
#pragma unroll
    for (int tt = 0; tt < kS1Tok; ++tt) acc[tt] = 0.f;
    for (int64_t i = j * a.g + int64_t(threadIdx.x) * 8; i < (j + 1) * a.g; i += kBlock * 8) {
#pragma unroll
      for (int tt = 0; tt < kS1Tok; ++tt) {
        if (tt < ntok) {
          const uint4 xv = *reinterpret_cast<const uint4*>(a.x + (m0 + tt) * a.ldx + i);
          acc[tt] += (bf16_lo(xv.x) + bf16_hi(xv.x)) + (bf16_lo(xv.y) + bf16_hi(xv.y)) +
                     (bf16_lo(xv.z) + bf16_hi(xv.z)) + (bf16_lo(xv.w) + bf16_hi(xv.w));
        }
      }
    }
#pragma unroll
    for (int tt = 0; tt < kS1Tok; ++tt) {
      const float v = seg_sum<64>(acc[tt]);
      if (lane == 0) red[wid][tt] = v;
    }
    __syncthreads();
    if (threadIdx.x < ntok) {
      const int tt = threadIdx.x;
      float v = red[0][tt];
      for (int w = 1; w < kWaves; ++w) v += red[w][tt];
      a.xs[(m0 + tt) * ngrp + j] = v;
    }
    return;
  }
  const bool core = k < a.rc;
  const int8_t* crow = core ? a.cv + k * a.d : a.cb + (k - a.rc) * a.d;
  const int64_t grp = core ? a.gv : a.gb;
  const uint16_t* srow = core ? a.sv + k * (a.d / a.gv) : a.sb + (k - a.rc) * (a.d / a.gb);
  const int ntok = int(a.M - m0 < kS1Tok ? a.M - m0 : kS1Tok);
  float acc[kS1Tok];
#pragma unroll
  for (int j = 0; j < kS1Tok; ++j) acc[j] = 0.f;
#pragma unroll 4
  for (int64_t i = int64_t(threadIdx.x) * 8; i < a.d; i += kBlock * 8) {
    const uint2 cw = *reinterpret_cast<const uint2*>(crow + i);
    const float s = f16_to_f32(srow[i / grp]);
    float w[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      w[j] = float(int8_t(cw.x >> (8 * j))) * s;
      w[4 + j] = float(int8_t(cw.y >> (8 * j))) * s;
    }
#pragma unroll
    for (int tt = 0; tt < kS1Tok; ++tt) {
      if (tt < ntok) {
        const uint4 xv = *reinterpret_cast<const uint4*>(a.x + (m0 + tt) * a.ldx + i);
        const uint32_t xs[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[tt] = fmaf(bf16_lo(xs[j]), w[2 * j], acc[tt]);
          acc[tt] = fmaf(bf16_hi(xs[j]), w[2 * j + 1], acc[tt]);
        }
      }
    }
  }
#pragma unroll
  for (int tt = 0; tt < kS1Tok; ++tt) {
    const float v = seg_sum<64>(acc[tt]);
    if (lane == 0) red[wid][tt] = v;
  }
  __syncthreads();
  if (threadIdx.x < ntok) {
    const int tt = threadIdx.x;
    float v = red[0][tt];
    for (int w = 1; w < kWaves; ++w) v += red[w][tt];
    a.t[(m0 + tt) * R + k] = v;
  }
}

// ------------------------------------------------------------ decode GEMV
// Lanes are split into segments of LPR lanes; a segment owns one vocabulary
// row at a time and walks along d in 16-byte chunks (32 codes), LPR chunks
// per iteration, so each segment load is LPR * 16 contiguous bytes.  A wave
// step covers kRowsPerStep rows per segment (WR rows in all).  Waves get
// contiguous, balanced ranges of steps (persistent grid).  x, the chunk
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
  const float* t;  // [M, rc + rr]
  int64_t tok0;    // first token of this pass
  int64_t V;
  int d, g, rc, rr;
  int gshift;      // log2(g / 32) when g is a power of two, else -1
  int vec_exp;     // expansion codes loaded as one dword per lane (see ExpOps)
  int64_t cu_stride, ca_stride, su_stride, sa_stride;  // 0 for an absent factor
  int nit;         // iterations along d: (d / 32) / LPR
  int64_t nsteps;  // ceil(V / rows per wave step)
  void* out;
  int64_t ldo;
  int out_bf16;
  // fused CE
  const void* tgt;
  int tgt64;
  float2* part;    // [M, n_part]
  int64_t n_part;
  float* tgt_logit;  // [M]
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
  uint32_t c[RB][KD];   // four int8 codes
  uint32_t s[RB][KD];   // fp16 bit pattern of the row scale
};

template <int LPR>
struct ExpLanes {
  static constexpr int KD = LPR >= 64 ? 1 : 2;
};

// acc += scale * (codes . t) over the lane's dwords of each row.
template <int TOK, int RB, int KD, int LPR>
__device__ __forceinline__ void apply_expansion(float (&acc)[RB][TOK], const ExpOps<RB, KD>& e,
                                                const float* st, int R, int sl) {
  const int R4 = R / 4;
#pragma unroll
  for (int kd = 0; kd < KD; ++kd) {
    const int q = sl + kd * LPR;
    const bool valid = q < R4;
    const int qq = valid ? q : 0;
#pragma unroll
    for (int tt = 0; tt < TOK; ++tt) {
      const float4 t4 = *reinterpret_cast<const float4*>(st + tt * R + 4 * qq);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const uint32_t u = e.c[rb][kd];
        float du = float(int8_t(u)) * t4.x;
        du = fmaf(float(int8_t(u >> 8)), t4.y, du);
        du = fmaf(float(int8_t(u >> 16)), t4.z, du);
        du = fmaf(float(int8_t(u >> 24)), t4.w, du);
        const float sc = valid ? f16_to_f32(uint16_t(e.s[rb][kd])) : 0.f;
        acc[rb][tt] = fmaf(sc, du, acc[rb][tt]);
      }
    }
  }
}

// One d-iteration of a step: RB rows x one 16-byte chunk per lane.
template <int TOK, int RB>
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
    const float s = f16_to_f32(uint16_t(sc[rb]));
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

// Per-lane softmax state of the fused CE epilogue.
template <int TOK>
struct CeState {
  float mx[TOK], se[TOK];
  int64_t y[TOK];
};

// End of a step: add the rank-r expansions of the lane's rows, reduce over
// the segment and store the logits (or fold them into the softmax state).
// Row rb of the lane is row0 + min(seg + rb * SEG, lim).
template <int TOK, int LPR, int RB, bool CE, bool EXPAND>
__device__ __forceinline__ void gemv_epilogue(float (&acc)[RB][TOK], const GemvArgs& a,
                                              int64_t row0, uint32_t lim, int seg, int sl,
                                              int lane, int my_row, bool writer,
                                              const float* st, CeState<TOK>& ce) {
  constexpr int SEG = 64 / LPR;
  const int R = a.rc + a.rr;
#pragma unroll
  for (int rb = 0; rb < RB && EXPAND; ++rb) {
    uint32_t r = uint32_t(seg + rb * SEG);
    r = r < lim ? r : lim;
    const int64_t v = row0 + r;
    if (a.rc) {
      const float su = f16_to_f32(a.su[v]);
      for (int k = sl; k < a.rc; k += LPR) {
        const float u = su * float(a.cu[v * a.rc + k]);
#pragma unroll
        for (int tt = 0; tt < TOK; ++tt) acc[rb][tt] = fmaf(u, st[tt * R + k], acc[rb][tt]);
      }
    }
    if (a.rr) {
      const float sa = f16_to_f32(a.sa[v]);
      for (int k = sl; k < a.rr; k += LPR) {
        const float u = sa * float(a.ca[v * a.rr + k]);
#pragma unroll
        for (int tt = 0; tt < TOK; ++tt)
          acc[rb][tt] = fmaf(u, st[tt * R + a.rc + k], acc[rb][tt]);
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
    if (store) {
      if constexpr (!CE) {
        const int64_t o = (a.tok0 + tt) * a.ldo + v;
        if (a.out_bf16)
          reinterpret_cast<uint16_t*>(a.out)[o] = f32_to_bf16_rne(l);
        else
          reinterpret_cast<float*>(a.out)[o] = l;
      } else {
        if (l > ce.mx[tt]) {
          ce.se[tt] = ce.se[tt] * fast_exp(ce.mx[tt] - l) + 1.f;
          ce.mx[tt] = l;
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
template <int TOK, int LPR, bool CE>
__global__ __launch_bounds__(kBlock)
__attribute__((amdgpu_waves_per_eu(TOK == 1 ? (LPR >= 64 ? ARCHEAD_GEMV_WAVES : 2) : 1)))
void k_gemv(GemvArgs a) {
  constexpr int SEG = 64 / LPR;              // rows in flight per wave
  constexpr int RB = LPR < kRowsPerStep ? LPR : kRowsPerStep;
  constexpr int WR = RB * SEG;               // rows per wave step
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ float2 red[kWaves][TOK];

  const int d = a.d;
  const int C = d / 32;                      // 16-byte chunks per row
  const int R = a.rc + a.rr;
  uint16_t* sx = reinterpret_cast<uint16_t*>(smem);          // [TOK][d]
  float* sxb = reinterpret_cast<float*>(sx + TOK * d);        // [TOK][C]
  float* st = sxb + TOK * C;                                  // [TOK][R]

  {
    const int x8 = d / 8;   // 16-byte units per token: unit u = chunk u/4, part u%4
    for (int i = threadIdx.x; i < TOK * x8; i += kBlock) {
      const int tt = i / x8, u = i - tt * x8;
      reinterpret_cast<uint4*>(sx)[(tt * 4 + (u & 3)) * C + (u >> 2)] =
          *reinterpret_cast<const uint4*>(a.x + (a.tok0 + tt) * a.ldx + u * 8);
    }
    for (int i = threadIdx.x; i < TOK * R; i += kBlock) {
      const int tt = i / R;
      st[i] = a.t[(a.tok0 + tt) * R + (i - tt * R)];
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
  }

  const int lane = threadIdx.x & 63;
  const int seg = lane / LPR, sl = lane % LPR;
  // Steps are dealt out grid-stride (wave gw takes steps gw, gw + W, ...), so
  // at any moment the whole grid streams one compact window of the head.
  const int64_t W = int64_t(gridDim.x) * kWaves;
  const int wid = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int64_t gw = int64_t(blockIdx.x) * kWaves + wid;
  const uint32_t rowbytes = uint32_t(d) / 2;
  const uint32_t ngrp = uint32_t(d / a.g);
  const int my_row = row_of_lane<LPR, RB>(lane);   // row this lane ends up with
  const bool writer = (sl & (LPR / RB - 1)) == 0;
  // nibble-pair mask and bf16 128.0 bit pattern, held in registers
  const uint32_t kMask = __builtin_amdgcn_readfirstlane(0x000F000Fu);
  const uint32_t kMagic = __builtin_amdgcn_readfirstlane(0x43004300u);

  CeState<TOK> ce;
#pragma unroll
  for (int tt = 0; tt < TOK; ++tt) {
    ce.mx[tt] = -INFINITY;
    ce.se[tt] = 0.f;
    if constexpr (CE)
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
  const int64_t full_steps = a.vec_exp ? a.V / WR : 0;
  if (gw < full_steps) {
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
    const int rc4 = a.rc / 4, R4 = R / 4;
    auto load = [&](int64_t stp, int itx, uint4 (&q)[RB], uint32_t (&sc)[RB]) {
      const uint64_t cbytes = uint64_t(a.V - stp * WR) * rowbytes;
      const uint64_t sbytes = uint64_t(a.V - stp * WR) * ngrp * 2u;
      const __amdgpu_buffer_rsrc_t rc_ = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint8_t*>(a.codes + uint64_t(stp) * WR * rowbytes), 0,
          int(cbytes < 0xffffffffull ? cbytes : 0xffffffffull), kBufferWord3);
      const __amdgpu_buffer_rsrc_t rs_ = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint16_t*>(a.rs + uint64_t(stp) * WR * ngrp), 0,
          int(sbytes < 0xffffffffull ? sbytes : 0xffffffffull), kBufferWord3);
      const uint32_t c = uint32_t(itx * LPR + sl);
      const uint32_t grp = a.gshift >= 0 ? (c >> a.gshift) : (c * 32u) / uint32_t(a.g);
      const int itoff = itx * LPR * 16;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(
            rc_, int(voff), int(uint32_t(rb * SEG) * rowbytes) + itoff, kLoadStream);
        q[rb] = make_uint4(v.x, v.y, v.z, v.w);
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        sc[rb] = __builtin_amdgcn_raw_buffer_load_b16(
            rs_, int((svoff + grp) * 2u), int(uint32_t(rb * SEG) * ngrp * 2u), 0);
    };
    // expansion operands of step stp (one buffer: the next step's operands
    // are requested right after the current step's have been applied)
    auto load_exp = [&](int64_t stp, ExpOps<RB, KD>& e) {
      const int64_t v0 = stp * WR + seg;
#pragma unroll
      for (int kd = 0; kd < KD; ++kd) {
        int q = sl + kd * LPR;
        q = q < R4 ? q : 0;
        const bool isu = q < rc4;
        const int8_t* cb = isu ? a.cu + 4 * q : a.ca + 4 * (q - rc4);
        const int64_t cs = isu ? a.cu_stride : a.ca_stride;
        const uint16_t* sp = isu ? a.su : a.sa;
        const int64_t ss = isu ? a.su_stride : a.sa_stride;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const int64_t v = v0 + rb * SEG;
          e.c[rb][kd] = *reinterpret_cast<const uint32_t*>(cb + v * cs);
          e.s[rb][kd] = sp[v * ss];
        }
      }
    };
    uint4 q[NB][RB];
    uint32_t sc[NB][RB];
    ExpOps<RB, KD> e;
    const int64_t last_step = gw + ((full_steps - 1 - gw) / W) * W;
    auto advance = [&](int64_t& st, int& itv) {
      if (++itv == a.nit) { itv = 0; st += W; }
    };
    int64_t cstep = gw, lstep = gw;   // compute and load cursors
    int cit = 0, lit = 0;
#pragma unroll
    for (int j = 0; j < kPD; ++j) {
      const bool ok = lstep < full_steps;
      load(ok ? lstep : last_step, ok ? lit : a.nit - 1, q[j], sc[j]);
      advance(lstep, lit);
    }
    load_exp(cstep, e);
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
      if (cit == 0) apply_expansion<TOK, RB, KD, LPR>(acc, e, st, R, sl);
      int64_t nstep = cstep;
      int nit = cit;
      advance(nstep, nit);
      const bool more = nstep < full_steps;
      if (nit == 0) load_exp(more ? nstep : cstep, e);
      gemv_chunk<TOK, RB>(acc, q[j], sc[j], sx, sxb, d, C, cit * LPR + sl, kMask, kMagic);
      if (cit == a.nit - 1)
        gemv_epilogue<TOK, LPR, RB, CE, false>(acc, a, cstep * WR, uint32_t(WR - 1), seg, sl,
                                               lane, my_row, writer, st, ce);
      cstep = nstep;
      cit = nit;
      done = !more;
    };
    while (true) {
      body(std::integral_constant<int, 0>{});
      if (done) break;
      body(std::integral_constant<int, 1>{});
      if (done) break;
      if constexpr (NB > 2) {
        body(std::integral_constant<int, 2 % NB>{});
        if (done) break;
      }
      if constexpr (NB > 3) {
        body(std::integral_constant<int, 3 % NB>{});
        if (done) break;
      }
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
        sc[rb] = sbase[uint64_t(r) * ngrp + grp];
      }
      gemv_chunk<TOK, RB>(acc, q, sc, sx, sxb, d, C, int(c), kMask, kMagic);
    }
    gemv_epilogue<TOK, LPR, RB, CE, true>(acc, a, row0, lim, seg, sl, lane, my_row, writer, st,
                                          ce);
  }

  if constexpr (CE) {
#pragma unroll
    for (int tt = 0; tt < TOK; ++tt) {
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const float om = __shfl_xor(ce.mx[tt], off, 64);
        const float os = __shfl_xor(ce.se[tt], off, 64);
        lse_merge(ce.mx[tt], ce.se[tt], om, os);
      }
      if (lane == 0) red[wid][tt] = make_float2(ce.mx[tt], ce.se[tt]);
    }
    __syncthreads();
    if (threadIdx.x < TOK) {
      const int tt = threadIdx.x;
      float m = red[0][tt].x, s = red[0][tt].y;
      for (int w = 1; w < kWaves; ++w) lse_merge(m, s, red[w][tt].x, red[w][tt].y);
      a.part[(a.tok0 + tt) * a.n_part + blockIdx.x] = make_float2(m, s);
    }
  }
}

// ------------------------------------------------------------ prefill MFMA
// Tiled bf16 MFMA kernel for many tokens.  A workgroup owns a kTM x kTN tile
// (tokens x vocabulary rows); its four waves own 64 x 64 quarters, each a
// 4 x 4 grid of 16x16 MFMA tiles (v_mfma_f32_16x16x32_bf16: A lane l holds
// row l%16, k = 8 (l/16) .. +7; B likewise by column; D lane l holds rows
// 4 (l/16) .. +3 of column l%16).  The K loop runs over d in stages of KS
// elements staged in double-buffered LDS (rows padded so fragment reads are
// bank-conflict free).  Codes are unpacked to bf16 (136 + c) per wave; the
// MFMA of the first chunk of every scale group starts from -136 * (sum of x
// over the group), so the group partial is sum c x; the fp32 group scale then
// multiplies it into the accumulator.  The rank-r expansion runs as extra
// K-chunks with t split into three bf16 parts (hi + mid + lo = t to fp32
// precision) against the int8 codes (exact in bf16), scaled by s_U / s_A.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kTM = 128, kTN = 128;

struct MfmaArgs {
  const uint8_t* codes;
  const uint16_t* rs;
  const int8_t* cu;
  const uint16_t* su;
  const int8_t* ca;
  const uint16_t* sa;
  const uint16_t* x;
  int64_t ldx;
  const float* t;    // [M, rc + rr]
  const float* xs;   // [M, d/g]
  int64_t M, V;
  int d, g, rc, rr;
  int64_t n_vt, n_tiles, tiles_per_xcd;
  void* out;
  int64_t ldo;
  int out_bf16;
  const void* tgt;
  int tgt64;
  float2* part;      // [M, n_vt]
  float* tgt_logit;  // [M]
};

__device__ __forceinline__ bf16x8_t unpack8(uint32_t q, uint32_t kMask, uint32_t kMagic) {
  uint32_t p[4];
  p[0] = int4_pair<0>(q, kMask, kMagic);
  p[1] = int4_pair<1>(q, kMask, kMagic);
  p[2] = int4_pair<2>(q, kMask, kMagic);
  p[3] = int4_pair<3>(q, kMask, kMagic);
  return __builtin_bit_cast(bf16x8_t, p);
}

template <int KS, bool CE>
__global__ __launch_bounds__(kBlock) void k_mfma(MfmaArgs a) {
  constexpr int KC = KS / 32;            // MFMA K-chunks per stage
  constexpr int XROW = KS + 8;           // bf16 per LDS x row (16 bytes of padding)
  constexpr int CROW = KS / 2 + 16;      // bytes per LDS code row (16 bytes of padding)
  constexpr int XBUF = kTM * XROW * 2;   // bytes of one x buffer
  constexpr int CBUF = kTN * CROW;       // bytes of one code buffer
  constexpr int TROW = 32 + 4;           // floats per LDS t row (expansion)
  constexpr int EROW = 32 + 8;           // bf16 per LDS expansion-code row
  constexpr int TBYTES = kTM * TROW * 4, EBYTES = kTN * EROW * 2;   // expansion staging
  constexpr int POOL = 2 * XBUF + 2 * CBUF > TBYTES + EBYTES ? 2 * XBUF + 2 * CBUF
                                                              : TBYTES + EBYTES;
  __shared__ __align__(16) unsigned char lds[POOL];
  __shared__ float sscale[2][kTN];
  __shared__ float sbias[2][kTM];
  __shared__ int64_t sy[kTM];
  __shared__ float2 sred[2][kTM];

  // tile: workgroups are dealt to the 8 XCDs round-robin; give each XCD a
  // contiguous run of tiles (vocabulary tiles fastest) so concurrent tiles on
  // one XCD share the same token rows in its L2
  const int64_t b = blockIdx.x;
  const int64_t lin = (b % 8) * a.tiles_per_xcd + b / 8;
  if (lin >= a.n_tiles) return;
  const int64_t mt = lin / a.n_vt, vt = lin - mt * a.n_vt;
  const int64_t m0 = mt * kTM, v0 = vt * kTN;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 1, wn = wid & 1;
  const int lr = lane & 15, lq = lane >> 4;
  const uint32_t kMask = __builtin_amdgcn_readfirstlane(0x000F000Fu);
  const uint32_t kMagic = __builtin_amdgcn_readfirstlane(0x43004300u);
  const int ngrp = a.d / a.g;
  const int64_t rowbytes = a.d / 2;
  const int R = a.rc + a.rr;

  f32x4_t acc[4][4], D[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // ---- staging of one K stage: x [kTM x KS] bf16 and codes [kTN x KS/2]
  constexpr int XU = kTM * KS / 8 / kBlock;   // 16-byte x units per thread
  constexpr int CU = kTN * KS / 2 / 16;       // 16-byte code units in all
  uint4 rx[XU], rcd;
  auto gload = [&](int stage) {
    const int64_t k0 = int64_t(stage) * KS;
#pragma unroll
    for (int j = 0; j < XU; ++j) {
      const int u = tid + j * kBlock, r = u / (KS / 8), c8 = u % (KS / 8);
      const int64_t m = m0 + r < a.M ? m0 + r : a.M - 1;
      rx[j] = *reinterpret_cast<const uint4*>(a.x + m * a.ldx + k0 + 8 * c8);
    }
    if (tid < CU) {
      const int r = tid / (KS / 32), c16 = tid % (KS / 32);
      const int64_t v = v0 + r < a.V ? v0 + r : a.V - 1;
      rcd = *reinterpret_cast<const uint4*>(a.codes + v * rowbytes + k0 / 2 + 16 * c16);
    }
  };
  auto lstore = [&](int buf) {
    uint16_t* sx = reinterpret_cast<uint16_t*>(lds + buf * XBUF);
#pragma unroll
    for (int j = 0; j < XU; ++j) {
      const int u = tid + j * kBlock, r = u / (KS / 8), c8 = u % (KS / 8);
      *reinterpret_cast<uint4*>(sx + r * XROW + 8 * c8) = rx[j];
    }
    if (tid < CU) {
      const int r = tid / (KS / 32), c16 = tid % (KS / 32);
      *reinterpret_cast<uint4*>(lds + 2 * XBUF + buf * CBUF + r * CROW + 16 * c16) = rcd;
    }
  };
  // scale group j: scales of the tile's columns and -136 * xs of its rows
  float gsc = 0.f, gbi = 0.f;
  auto gload_group = [&](int j) {
    if (tid < kTN) {
      const int64_t v = v0 + tid < a.V ? v0 + tid : a.V - 1;
      gsc = f16_to_f32(a.rs[v * ngrp + j]);
    } else {
      const int r = tid - kTN;
      const int64_t m = m0 + r < a.M ? m0 + r : a.M - 1;
      gbi = -float(archead::kInt4Bias) * a.xs[m * ngrp + j];
    }
  };
  auto lstore_group = [&](int j) {
    if (tid < kTN) sscale[j & 1][tid] = gsc;
    else sbias[j & 1][tid - kTN] = gbi;
  };
  if (CE && tid < kTM) {
    const int64_t m = m0 + tid < a.M ? m0 + tid : a.M - 1;
    sy[tid] = a.tgt64 ? reinterpret_cast<const int64_t*>(a.tgt)[m]
                      : int64_t(reinterpret_cast<const int32_t*>(a.tgt)[m]);
  }

  const int nstage = a.d / KS;
  const int spg = a.g / KS;   // stages per scale group
  gload(0);
  gload_group(0);
  lstore(0);
  lstore_group(0);
  __syncthreads();

  for (int s = 0; s < nstage; ++s) {
    const int buf = s & 1, grp = s / spg;
    const bool gstart = s % spg == 0, gend = (s + 1) % spg == 0;
    if (s + 1 < nstage) {
      gload(s + 1);
      if ((s + 1) % spg == 0) gload_group((s + 1) / spg);
    }
    const uint16_t* sx = reinterpret_cast<const uint16_t*>(lds + buf * XBUF);
    const unsigned char* scd = lds + 2 * XBUF + buf * CBUF;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      bf16x8_t A[4], B[4];
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
        A[mi] = *reinterpret_cast<const bf16x8_t*>(sx + (64 * wm + 16 * mi + lr) * XROW +
                                                   kc * 32 + 8 * lq);
#pragma unroll
      for (int ni = 0; ni < 4; ++ni)
        B[ni] = unpack8(*reinterpret_cast<const uint32_t*>(
                            scd + (64 * wn + 16 * ni + lr) * CROW + kc * 16 + 4 * lq),
                        kMask, kMagic);
      if (gstart && kc == 0) {
#pragma unroll
        for (int mi = 0; mi < 4; ++mi) {
          const float* sb = sbias[grp & 1] + 64 * wm + 16 * mi + 4 * lq;
          const f32x4_t bias = {sb[0], sb[1], sb[2], sb[3]};
#pragma unroll
          for (int ni = 0; ni < 4; ++ni)
            D[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[mi], B[ni], bias, 0, 0, 0);
        }
      } else {
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
          for (int ni = 0; ni < 4; ++ni)
            D[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[mi], B[ni], D[mi][ni], 0, 0, 0);
      }
    }
    if (gend) {
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        const float sc = sscale[grp & 1][64 * wn + 16 * ni + lr];
#pragma unroll
        for (int mi = 0; mi < 4; ++mi) acc[mi][ni] += sc * D[mi][ni];
      }
    }
    if (s + 1 < nstage) {
      lstore(buf ^ 1);
      if ((s + 1) % spg == 0) lstore_group((s + 1) / spg);
    }
    __syncthreads();
  }

  // ---- rank-r expansion: two more "groups" (core U_c, correction A_w)
#pragma unroll 1
  for (int part = 0; part < 2; ++part) {
    const int r = part ? a.rr : a.rc;
    if (r == 0) continue;
    const int8_t* codes8 = part ? a.ca : a.cu;
    const uint16_t* rscale = part ? a.sa : a.su;
    const int toff = part ? a.rc : 0;
    const int nchunk = (r + 31) / 32;
#pragma unroll 1
    for (int c = 0; c < nchunk; ++c) {
      float* st = reinterpret_cast<float*>(lds);                       // [kTM][TROW]
      __bf16* se = reinterpret_cast<__bf16*>(lds + TBYTES);            // [kTN][EROW]
      for (int e = tid; e < kTM * 32; e += kBlock) {
        const int row = e >> 5, k = e & 31, kk = c * 32 + k;
        const int64_t m = m0 + row < a.M ? m0 + row : a.M - 1;
        st[row * TROW + k] = kk < r ? a.t[m * R + toff + kk] : 0.f;
      }
      for (int e = tid; e < kTN * 32; e += kBlock) {
        const int col = e >> 5, k = e & 31, kk = c * 32 + k;
        const int64_t v = v0 + col < a.V ? v0 + col : a.V - 1;
        se[col * EROW + k] = kk < r ? (__bf16)float(codes8[v * r + kk]) : (__bf16)0.f;
      }
      __syncthreads();
      bf16x8_t B[4];
#pragma unroll
      for (int ni = 0; ni < 4; ++ni)
        B[ni] = *reinterpret_cast<const bf16x8_t*>(se + (64 * wn + 16 * ni + lr) * EROW + 8 * lq);
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) {
        const float* tp = st + (64 * wm + 16 * mi + lr) * TROW + 8 * lq;
        bf16x8_t hi, mid, lo;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float v = tp[j];
          const __bf16 h = (__bf16)v;
          const float r1 = v - float(h);
          const __bf16 m_ = (__bf16)r1;
          hi[j] = h;
          mid[j] = m_;
          lo[j] = (__bf16)(r1 - float(m_));
        }
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          f32x4_t dd = c == 0 ? f32x4_t{0.f, 0.f, 0.f, 0.f} : D[mi][ni];
          dd = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hi, B[ni], dd, 0, 0, 0);
          dd = __builtin_amdgcn_mfma_f32_16x16x32_bf16(mid, B[ni], dd, 0, 0, 0);
          D[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lo, B[ni], dd, 0, 0, 0);
        }
      }
      __syncthreads();
    }
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) {
      const int64_t v = v0 + 64 * wn + 16 * ni + lr;
      const float sc = f16_to_f32(rscale[v < a.V ? v : a.V - 1]);
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) acc[mi][ni] += sc * D[mi][ni];
    }
  }

  // ---- epilogue
  if constexpr (!CE) {
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t m = m0 + 64 * wm + 16 * mi + 4 * lq + i;
        if (m >= a.M) continue;
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          const int64_t v = v0 + 64 * wn + 16 * ni + lr;
          if (v >= a.V) continue;
          const float l = acc[mi][ni][i];
          if (a.out_bf16)
            reinterpret_cast<uint16_t*>(a.out)[m * a.ldo + v] = f32_to_bf16_rne(l);
          else
            reinterpret_cast<float*>(a.out)[m * a.ldo + v] = l;
        }
      }
  } else {
    // per-row (max, sum exp) over this tile's valid columns; the 16 lanes of a
    // quarter-wave share rows, the two waves of a row half are merged in LDS
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rloc = 64 * wm + 16 * mi + 4 * lq + i;
        float mx = -INFINITY;
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          const int64_t v = v0 + 64 * wn + 16 * ni + lr;
          if (v < a.V) mx = fmaxf(mx, acc[mi][ni][i]);
        }
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
        float se = 0.f;
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          const int64_t v = v0 + 64 * wn + 16 * ni + lr;
          if (v < a.V) {
            se += fast_exp(acc[mi][ni][i] - mx);
            if (v == sy[rloc] && m0 + rloc < a.M) a.tgt_logit[m0 + rloc] = acc[mi][ni][i];
          }
        }
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) se += __shfl_xor(se, off, 64);
        if (lr == 0) sred[wn][rloc] = make_float2(mx, se);
      }
    __syncthreads();
    if (tid < kTM && m0 + tid < a.M) {
      float m_ = sred[0][tid].x, s_ = sred[0][tid].y;
      lse_merge(m_, s_, sred[1][tid].x, sred[1][tid].y);
      a.part[(m0 + tid) * a.n_vt + vt] = make_float2(m_, s_);
    }
  }
}

// ---------------------------------------------------------------- CE merge
// ce[m] = MX + ln S - l[m, y_m], combining the per-tile (max, sum exp) pairs
// in a fixed order (strided per thread, then a fixed tree) so the result is
// reproducible bit for bit.
__global__ __launch_bounds__(kBlock) void k_ce_merge(const float2* part, int64_t n_part,
                                                     const void* tgt, int tgt64,
                                                     const float* tgt_logit, int64_t V,
                                                     float* ce) {
  __shared__ float smx[kBlock], sse[kBlock];
  const int64_t m = blockIdx.x;
  float mx = -INFINITY, se = 0.f;
  for (int64_t p = threadIdx.x; p < n_part; p += kBlock) {
    const float2 q = part[m * n_part + p];
    lse_merge(mx, se, q.x, q.y);
  }
  smx[threadIdx.x] = mx;
  sse[threadIdx.x] = se;
  __syncthreads();
  for (int s = kBlock / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
      float a = smx[threadIdx.x], b = sse[threadIdx.x];
      lse_merge(a, b, smx[threadIdx.x + s], sse[threadIdx.x + s]);
      smx[threadIdx.x] = a;
      sse[threadIdx.x] = b;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const int64_t y = tgt64 ? reinterpret_cast<const int64_t*>(tgt)[m]
                            : int64_t(reinterpret_cast<const int32_t*>(tgt)[m]);
    ce[m] = (y >= 0 && y < V) ? smx[0] + logf(sse[0]) - tgt_logit[m] : NAN;
  }
}

__global__ __launch_bounds__(kBlock) void k_mean(const float* v, int64_t n, float* out) {
  __shared__ float s[kBlock];
  float acc = 0.f;
  for (int64_t i = threadIdx.x; i < n; i += kBlock) acc += v[i];
  s[threadIdx.x] = acc;
  __syncthreads();
  for (int k = kBlock / 2; k > 0; k >>= 1) {
    if (threadIdx.x < k) s[threadIdx.x] += s[threadIdx.x + k];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = s[0] / float(n);
}

// ------------------------------------------------------------ dispatch
using GemvFn = void (*)(GemvArgs);

template <int TOK, bool CE>
GemvFn gemv_by_lpr(int lpr) {
  switch (lpr) {
    case 1: return k_gemv<TOK, 1, CE>;
    case 2: return k_gemv<TOK, 2, CE>;
    case 4: return k_gemv<TOK, 4, CE>;
    case 8: return k_gemv<TOK, 8, CE>;
    case 16: return k_gemv<TOK, 16, CE>;
    case 32: return k_gemv<TOK, 32, CE>;
    default: return k_gemv<TOK, 64, CE>;
  }
}

template <bool CE>
GemvFn gemv_fn(int tok, int lpr) {
  switch (tok) {
    case 1: return gemv_by_lpr<1, CE>(lpr);
    case 2: return gemv_by_lpr<2, CE>(lpr);
    case 3: return gemv_by_lpr<3, CE>(lpr);
    default: return gemv_by_lpr<4, CE>(lpr);
  }
}

size_t gemv_lds_bytes(const archead_desc& d, int tok) {
  return size_t(tok) * (size_t(d.d) * 2 + size_t(d.d / 32) * 4 + size_t(d.r_c + d.r_r) * 4);
}

int64_t gemv_rows_per_step(const archead_desc& d) {
  const int lpr = archead::lanes_per_row(d.d);
  return int64_t(lpr < kRowsPerStep ? lpr : kRowsPerStep) * (64 / lpr);
}

archead_status hip_fail(hipError_t e, const char* what) {
  return archead::fail(ARCHEAD_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

namespace archead {

int64_t gemv_grid(const archead_handle* h, int tok, bool ce) {
  const int slot = (ce ? 8 : 0) + tok;
  archead_handle* mh = const_cast<archead_handle*>(h);
  int cached = mh->grid_cache[slot].load(std::memory_order_relaxed);
  const int64_t steps = (h->desc.V + gemv_rows_per_step(h->desc) - 1) / gemv_rows_per_step(h->desc);
  const int64_t max_blocks = (steps + kWaves - 1) / kWaves;
  if (cached <= 0) {
    const int lpr = lanes_per_row(h->desc.d);
    GemvFn fn = ce ? gemv_fn<true>(tok, lpr) : gemv_fn<false>(tok, lpr);
    int nb = 0;
    const size_t lds = gemv_lds_bytes(h->desc, tok);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, reinterpret_cast<const void*>(fn),
                                                     kBlock, lds) != hipSuccess ||
        nb <= 0)
      nb = 1;
    // a few resident workgroups per CU stream best; ARCHEAD_GEMV_BLOCKS_PER_CU
    // overrides the built-in choice (tuning only)
    int want = kGemvBlocksPerCu;
    if (const char* e = getenv("ARCHEAD_GEMV_BLOCKS_PER_CU")) want = atoi(e) > 0 ? atoi(e) : want;
    if (nb > want) nb = want;
    cached = nb * h->n_cu;
    mh->grid_cache[slot].store(cached, std::memory_order_relaxed);
  }
  return cached < max_blocks ? cached : max_blocks;
}

static size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

WsLayout ws_layout(const archead_handle* h, int64_t M, archead_op op) {
  WsLayout w;
  if (!h || M <= 0) return w;
  const archead_desc& d = h->desc;
  size_t off = 0;
  const bool gemv = use_gemv(h, M);
  w.t_off = off;
  off = align256(off + sizeof(float) * size_t(M) * size_t(d.r_c + d.r_r));
  w.xs_off = off;
  if (!gemv) off = align256(off + sizeof(float) * size_t(M) * size_t(d.d / d.g));
  if (op == ARCHEAD_OP_LOGITS_CE) {
    // GEMV: all CE passes share one grid (the smallest of the variants
    // used) so every token row of the partials has the same number of
    // slots.  MFMA: one slot per vocabulary tile.
    int64_t np = 0;
    if (gemv) {
      const int64_t full = M / 4, rem = M % 4;
      if (full) np = gemv_grid(h, 4, true);
      if (rem) { const int64_t g = gemv_grid(h, int(rem), true); np = (np == 0 || g < np) ? g : np; }
    } else {
      np = (d.V + kTN - 1) / kTN;
    }
    w.n_part = np;
    w.part_off = off;
    off = align256(off + 2 * sizeof(float) * size_t(M) * size_t(np));
    w.tgt_off = off;
    off = align256(off + sizeof(float) * size_t(M));
  }
  w.total = off;
  return w;
}

}  // namespace archead

using namespace archead;

namespace {

archead_status check_call(const archead_handle* h, const void* x, int64_t M, int64_t ldx,
                          const void* ws, size_t ws_bytes, archead_op op) {
  if (!h) return fail(ARCHEAD_E_INVALID_ARG, "handle is NULL");
  if (M < 0) return fail(ARCHEAD_E_INVALID_ARG, "M = %lld < 0", (long long)M);
  if (M == 0) return ARCHEAD_OK;
  if (M > (int64_t(1) << 24)) return fail(ARCHEAD_E_UNSUPPORTED, "M must be <= 2^24");
  if (!x) return fail(ARCHEAD_E_INVALID_ARG, "x is NULL");
  if (ldx < h->desc.d) return fail(ARCHEAD_E_INVALID_ARG, "ldx < d");
  if (!aligned(x, 16) || ldx % 8) return fail(ARCHEAD_E_MISALIGNED, "x must be 16-byte aligned with ldx %% 8 == 0");
  const size_t need = ws_layout(h, M, op).total;
  if (ws_bytes < need) return fail(ARCHEAD_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  if (need && !ws) return fail(ARCHEAD_E_INVALID_ARG, "workspace is NULL");
  if (!aligned(ws, 256)) return fail(ARCHEAD_E_MISALIGNED, "workspace must be 256-byte aligned");
  return ARCHEAD_OK;
}

archead_status launch_stage1(const archead_handle* h, const void* x, int64_t M, int64_t ldx,
                             float* t, float* xs, hipStream_t s) {
  const archead_desc& d = h->desc;
  const int64_t R = d.r_c + d.r_r;
  const int64_t nx = xs ? d.d / d.g : 0;   // extra workgroups for the group sums
  if (R + nx == 0) return ARCHEAD_OK;
  Stage1Args a;
  a.x = static_cast<const uint16_t*>(x);
  a.ldx = ldx; a.M = M; a.d = d.d;
  a.cv = static_cast<const int8_t*>(h->ptrs.core_v);
  a.sv = static_cast<const uint16_t*>(h->ptrs.core_v_scale);
  a.gv = d.r_c ? d.g_v : d.d; a.rc = d.r_c;
  a.cb = static_cast<const int8_t*>(h->ptrs.corr_b);
  a.sb = static_cast<const uint16_t*>(h->ptrs.corr_b_scale);
  a.gb = d.r_r ? d.g_b : d.d; a.rr = d.r_r;
  a.t = t;
  a.xs = xs;
  a.g = d.g;
  for (int64_t m0 = 0; m0 < M; m0 += kMaxGridY * kS1Tok) {
    const int64_t rest = M - m0;
    const int64_t mblocks = (rest < kMaxGridY * kS1Tok ? rest + kS1Tok - 1 : kMaxGridY * kS1Tok) / kS1Tok;
    a.mbase = m0;
    hipLaunchKernelGGL(k_stage1, dim3(unsigned(R + nx), unsigned(mblocks)), dim3(kBlock), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "stage-1 launch");
  }
  return ARCHEAD_OK;
}

GemvArgs gemv_args(const archead_handle* h, const void* x, int64_t ldx, const float* t) {
  const archead_desc& d = h->desc;
  GemvArgs a;
  memset(&a, 0, sizeof a);
  a.codes = static_cast<const uint8_t*>(h->ptrs.res_codes);
  a.rs = static_cast<const uint16_t*>(h->ptrs.res_scales);
  a.cu = static_cast<const int8_t*>(h->ptrs.core_u);
  a.su = static_cast<const uint16_t*>(h->ptrs.core_u_scale);
  a.ca = static_cast<const int8_t*>(h->ptrs.corr_a);
  a.sa = static_cast<const uint16_t*>(h->ptrs.corr_a_scale);
  a.x = static_cast<const uint16_t*>(x);
  a.ldx = ldx;
  a.t = t;
  a.V = d.V; a.d = int(d.d); a.g = int(d.g); a.rc = int(d.r_c); a.rr = int(d.r_r);
  const int64_t cpg = d.g / 32;
  a.gshift = (cpg & (cpg - 1)) == 0 ? __builtin_ctzll(uint64_t(cpg)) : -1;
  const int lpr = lanes_per_row(d.d);
  const int kd = lpr >= 64 ? 1 : 2;   // ExpLanes<LPR>::KD
  a.vec_exp = d.r_c % 4 == 0 && d.r_r % 4 == 0 && (d.r_c + d.r_r) / 4 <= int64_t(kd) * lpr &&
              (d.r_c == 0 || aligned(h->ptrs.core_u, 4)) &&
              (d.r_r == 0 || aligned(h->ptrs.corr_a, 4));
  // an absent factor reads the (valid, 16-byte aligned) residual buffers with
  // stride 0 instead; its contribution is masked to zero in the kernel
  a.cu_stride = d.r_c; a.su_stride = d.r_c ? 1 : 0;
  a.ca_stride = d.r_r; a.sa_stride = d.r_r ? 1 : 0;
  if (!d.r_c) { a.cu = reinterpret_cast<const int8_t*>(a.codes); a.su = a.rs; }
  if (!d.r_r) { a.ca = reinterpret_cast<const int8_t*>(a.codes); a.sa = a.rs; }
  const int64_t wr = gemv_rows_per_step(d);
  a.nsteps = (d.V + wr - 1) / wr;
  a.nit = int((d.d / 32) / lanes_per_row(d.d));
  return a;
}

// One launch per group of up to 4 tokens.  forced_grid > 0 fixes the grid
// (the CE passes, whose partials are indexed by workgroup).
archead_status launch_gemv_passes(const archead_handle* h, GemvArgs a, int64_t M, bool ce,
                                  int64_t forced_grid, hipStream_t s) {
  const int lpr = lanes_per_row(h->desc.d);
  // timing events (if set) are attached to the first and last dispatch
  // packets themselves, so they bracket exactly the kernel execution
  hipEvent_t ev0 = static_cast<hipEvent_t>(h->ev_start.load(std::memory_order_relaxed));
  hipEvent_t ev1 = static_cast<hipEvent_t>(h->ev_stop.load(std::memory_order_relaxed));
  for (int64_t m0 = 0; m0 < M; m0 += 4) {
    const int tok = int(M - m0 < 4 ? M - m0 : 4);
    GemvFn fn = ce ? gemv_fn<true>(tok, lpr) : gemv_fn<false>(tok, lpr);
    const int64_t grid = forced_grid > 0 ? forced_grid : gemv_grid(h, tok, ce);
    a.tok0 = m0;
    const size_t lds = gemv_lds_bytes(h->desc, tok);
    if (lds > 65536) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
      if (e != hipSuccess) return hip_fail(e, "LDS size attribute");
    }
    void* args[] = {&a};
    const bool first = m0 == 0, last = m0 + 4 >= M;
    hipError_t e = hipExtLaunchKernel(reinterpret_cast<const void*>(fn), dim3(unsigned(grid)),
                                      dim3(kBlock), args, lds, s, first ? ev0 : nullptr,
                                      last ? ev1 : nullptr, 0);
    if (e != hipSuccess) return hip_fail(e, "GEMV launch");
  }
  return ARCHEAD_OK;
}

MfmaArgs mfma_args(const archead_handle* h, const void* x, int64_t M, int64_t ldx,
                   const float* t, const float* xs) {
  const archead_desc& d = h->desc;
  MfmaArgs a;
  memset(&a, 0, sizeof a);
  a.codes = static_cast<const uint8_t*>(h->ptrs.res_codes);
  a.rs = static_cast<const uint16_t*>(h->ptrs.res_scales);
  a.cu = static_cast<const int8_t*>(h->ptrs.core_u);
  a.su = static_cast<const uint16_t*>(h->ptrs.core_u_scale);
  a.ca = static_cast<const int8_t*>(h->ptrs.corr_a);
  a.sa = static_cast<const uint16_t*>(h->ptrs.corr_a_scale);
  a.x = static_cast<const uint16_t*>(x);
  a.ldx = ldx;
  a.t = t;
  a.xs = xs;
  a.M = M; a.V = d.V;
  a.d = int(d.d); a.g = int(d.g); a.rc = int(d.r_c); a.rr = int(d.r_r);
  a.n_vt = (d.V + kTN - 1) / kTN;
  a.n_tiles = a.n_vt * ((M + kTM - 1) / kTM);
  a.tiles_per_xcd = (a.n_tiles + 7) / 8;
  return a;
}

archead_status launch_mfma(const archead_handle* h, MfmaArgs a, bool ce, hipStream_t s) {
  using Fn = void (*)(MfmaArgs);
  const bool k64 = a.g % 64 == 0;
  Fn fn = ce ? (k64 ? k_mfma<64, true> : k_mfma<32, true>)
             : (k64 ? k_mfma<64, false> : k_mfma<32, false>);
  hipEvent_t ev0 = static_cast<hipEvent_t>(h->ev_start.load(std::memory_order_relaxed));
  hipEvent_t ev1 = static_cast<hipEvent_t>(h->ev_stop.load(std::memory_order_relaxed));
  void* args[] = {&a};
  hipError_t e = hipExtLaunchKernel(reinterpret_cast<const void*>(fn),
                                    dim3(unsigned(8 * a.tiles_per_xcd)), dim3(kBlock), args, 0,
                                    s, ev0, ev1, 0);
  return e == hipSuccess ? ARCHEAD_OK : hip_fail(e, "MFMA launch");
}

}  // namespace

extern "C" {

archead_status archead_create(const archead_desc* desc, const archead_ptrs* ptrs,
                              archead_handle** out) {
  clear_error();
  if (!out) return fail(ARCHEAD_E_INVALID_ARG, "out is NULL");
  *out = nullptr;
  archead_status st = archead_validate_desc(desc);
  if (st != ARCHEAD_OK) return st;
  if (!ptrs) return fail(ARCHEAD_E_INVALID_ARG, "ptrs is NULL");
  const archead_desc& d = *desc;
  if (!ptrs->res_codes || !ptrs->res_scales)
    return fail(ARCHEAD_E_INVALID_ARG, "res_codes and res_scales are required");
  if (d.r_c && (!ptrs->core_u || !ptrs->core_u_scale || !ptrs->core_v || !ptrs->core_v_scale))
    return fail(ARCHEAD_E_INVALID_ARG, "r_c > 0 needs core_u, core_u_scale, core_v, core_v_scale");
  if (d.r_r && (!ptrs->corr_a || !ptrs->corr_a_scale || !ptrs->corr_b || !ptrs->corr_b_scale))
    return fail(ARCHEAD_E_INVALID_ARG, "r_r > 0 needs corr_a, corr_a_scale, corr_b, corr_b_scale");
  if (!aligned(ptrs->res_codes, 16)) return fail(ARCHEAD_E_MISALIGNED, "res_codes must be 16-byte aligned");
  const void* f16s[] = {ptrs->res_scales, ptrs->core_u_scale, ptrs->core_v_scale,
                        ptrs->corr_a_scale, ptrs->corr_b_scale};
  for (const void* p : f16s)
    if (p && !aligned(p, 2)) return fail(ARCHEAD_E_MISALIGNED, "fp16 scales must be 2-byte aligned");
  if ((ptrs->core_v && !aligned(ptrs->core_v, 16)) || (ptrs->corr_b && !aligned(ptrs->corr_b, 16)))
    return fail(ARCHEAD_E_MISALIGNED, "core_v and corr_b must be 16-byte aligned");

  int dev = -1, ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || ndev <= 0)
    return fail(ARCHEAD_E_UNSUPPORTED, "no HIP device");
  if (hipGetDevice(&dev) != hipSuccess) return fail(ARCHEAD_E_UNSUPPORTED, "no current HIP device");
  hipDeviceProp_t prop;
  hipError_t e = hipGetDeviceProperties(&prop, dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
  if (strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(ARCHEAD_E_UNSUPPORTED, "device %d is %s, this library is built for gfx950", dev,
                prop.gcnArchName);
  archead_handle* h = new (std::nothrow) archead_handle();
  if (!h) return fail(ARCHEAD_E_INVALID_ARG, "out of host memory");
  h->desc = d;
  h->ptrs = *ptrs;
  h->device = dev;
  h->n_cu = prop.multiProcessorCount;
  h->gemv_max_m.store(kDefaultGemvMaxM);
  for (auto& c : h->grid_cache) c.store(0);
  h->ev_start.store(nullptr);
  h->ev_stop.store(nullptr);
  *out = h;
  return ARCHEAD_OK;
}

void archead_destroy(archead_handle* h) { delete h; }

size_t archead_workspace_bytes(const archead_handle* h, int64_t M, archead_op op) {
  if (!h || M <= 0) return 0;
  return ws_layout(h, M, op).total;
}

archead_status archead_logits(const archead_handle* h, const void* x, int64_t M, int64_t ldx,
                              void* out, archead_dtype out_dtype, int64_t ldo, void* ws,
                              size_t ws_bytes, void* stream) {
  clear_error();
  archead_status st = check_call(h, x, M, ldx, ws, ws_bytes, ARCHEAD_OP_LOGITS);
  if (st != ARCHEAD_OK || M == 0) return st;
  if (!out) return fail(ARCHEAD_E_INVALID_ARG, "out is NULL");
  if (out_dtype != ARCHEAD_F32 && out_dtype != ARCHEAD_BF16)
    return fail(ARCHEAD_E_INVALID_ARG, "out_dtype must be ARCHEAD_F32 or ARCHEAD_BF16");
  if (ldo < h->desc.V) return fail(ARCHEAD_E_INVALID_ARG, "ldo < V");
  if (!aligned(out, out_dtype == ARCHEAD_F32 ? 4 : 2))
    return fail(ARCHEAD_E_MISALIGNED, "out is not aligned to its element size");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const WsLayout w = ws_layout(h, M, ARCHEAD_OP_LOGITS);
  float* t = reinterpret_cast<float*>(static_cast<char*>(ws) + w.t_off);
  if (!use_gemv(h, M)) {
    float* xs = reinterpret_cast<float*>(static_cast<char*>(ws) + w.xs_off);
    st = launch_stage1(h, x, M, ldx, t, xs, s);
    if (st != ARCHEAD_OK) return st;
    MfmaArgs a = mfma_args(h, x, M, ldx, t, xs);
    a.out = out;
    a.ldo = ldo;
    a.out_bf16 = out_dtype == ARCHEAD_BF16;
    return launch_mfma(h, a, false, s);
  }
  st = launch_stage1(h, x, M, ldx, t, nullptr, s);
  if (st != ARCHEAD_OK) return st;
  GemvArgs a = gemv_args(h, x, ldx, t);
  a.out = out;
  a.ldo = ldo;
  a.out_bf16 = out_dtype == ARCHEAD_BF16;
  return launch_gemv_passes(h, a, M, false, 0, s);
}

archead_status archead_logits_ce(const archead_handle* h, const void* x, int64_t M, int64_t ldx,
                                 const void* targets, archead_dtype tgt_dtype, float* ce,
                                 float* mean_ce, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  archead_status st = check_call(h, x, M, ldx, ws, ws_bytes, ARCHEAD_OP_LOGITS_CE);
  if (st != ARCHEAD_OK || M == 0) return st;
  if (!targets || !ce) return fail(ARCHEAD_E_INVALID_ARG, "targets and ce are required");
  if (tgt_dtype != ARCHEAD_I32 && tgt_dtype != ARCHEAD_I64)
    return fail(ARCHEAD_E_INVALID_ARG, "tgt_dtype must be ARCHEAD_I32 or ARCHEAD_I64");
  if (!aligned(targets, tgt_dtype == ARCHEAD_I64 ? 8 : 4) || !aligned(ce, 4) ||
      (mean_ce && !aligned(mean_ce, 4)))
    return fail(ARCHEAD_E_MISALIGNED, "targets / ce / mean_ce misaligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const WsLayout w = ws_layout(h, M, ARCHEAD_OP_LOGITS_CE);
  char* base = static_cast<char*>(ws);
  float* t = reinterpret_cast<float*>(base + w.t_off);
  float2* part = reinterpret_cast<float2*>(base + w.part_off);
  float* tl = reinterpret_cast<float*>(base + w.tgt_off);
  const int64_t n_part = w.n_part;
  if (!use_gemv(h, M)) {
    float* xs = reinterpret_cast<float*>(base + w.xs_off);
    st = launch_stage1(h, x, M, ldx, t, xs, s);
    if (st != ARCHEAD_OK) return st;
    MfmaArgs a = mfma_args(h, x, M, ldx, t, xs);
    a.tgt = targets;
    a.tgt64 = tgt_dtype == ARCHEAD_I64;
    a.part = part;
    a.tgt_logit = tl;
    st = launch_mfma(h, a, true, s);
  } else {
    st = launch_stage1(h, x, M, ldx, t, nullptr, s);
    if (st != ARCHEAD_OK) return st;
    GemvArgs a = gemv_args(h, x, ldx, t);
    a.tgt = targets;
    a.tgt64 = tgt_dtype == ARCHEAD_I64;
    a.part = part;
    a.n_part = n_part;
    a.tgt_logit = tl;
    st = launch_gemv_passes(h, a, M, true, n_part, s);
  }
  if (st != ARCHEAD_OK) return st;
  hipLaunchKernelGGL(k_ce_merge, dim3(unsigned(M)), dim3(kBlock), 0, s, part, n_part, targets,
                     int(tgt_dtype == ARCHEAD_I64), tl, h->desc.V, ce);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "CE merge launch");
  if (mean_ce) {
    hipLaunchKernelGGL(k_mean, dim3(1), dim3(kBlock), 0, s, ce, M, mean_ce);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "mean launch");
  }
  return ARCHEAD_OK;
}

}  // extern "C"
