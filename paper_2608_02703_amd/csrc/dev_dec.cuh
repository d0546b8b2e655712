// The MFMA decode kernel template (k_dec).
#pragma once

#include "dev_common.cuh"

namespace {

// ------------------------------------------------------------ decode: MFMA
// Decode-shaped kernel for up to 16 tokens per pass: the packed head is
// streamed once per pass while bf16 MFMAs (v_mfma_f32_16x16x32_bf16) do the
// dot products, so the vector ALUs only unpack codes and apply scales, and
// the cost per pass is the same for 1 and for 16 tokens.
//
// A wave owns units of 16 vocabulary rows (grid-stride over the units, every
// wave the same number but for the last round).  Lane l holds row j = l % 16
// of the unit and quarter q = l / 16.  A unit is walked in iterations:
//  * one per residual group G (GW = g / 32 code words per lane): lane (j, q)
//    loads words q GW .. q GW + GW - 1 of group G of its row, MFMA kc takes
//    word q GW + kc, i.e. the 8 elements G g + 8 (q GW + kc) .. +7, whose
//    INT4 codes unpack to the bf16 values 136 + c (the same element order as
//    the x fragment read from LDS).  The first MFMA's accumulator input is
//    the group's offset bias -136 * (sum of x over the group), so the chain
//    yields the group partial sum c x; the fp16 group scale multiplies it
//    into the running fp32 total.  Groups of 64 are loaded in pairs (4 words
//    per lane, as for g = 128) and each group of a pair gets its own chain,
//    fed the pair's code fragments with the other group's lanes zeroed.
//  * then the rank-r expansion in K-chunks of 32 rank dimensions (U_c part
//    first, then A_w; each zero-padded to whole chunks): lane (j, q) loads
//    the int8 codes of dims 8q .. 8q+7 of each chunk of its row, converts
//    them exactly to bf16, and three bf16 MFMAs (v_mfma_f32_16x16x32_bf16)
//    per chunk multiply them with t held in LDS as three bf16 parts
//    hi = bf16(t), mid = bf16(t - hi), lo = bf16(t - hi - mid), whose sum is
//    t to fp32 precision; the row scale s_U or s_A multiplies the result
//    into the total.
// Output lane (j, q) holds tokens 4q .. 4q+3 of row j.
//
// Stage 1 (t = x V_c^T, x B_w^T) runs in the same launch: the first
// n_prod_blocks workgroups compute one rank row per wave and publish each
// value together with the call's epoch in one 64-bit store.  The other
// workgroups need t only at their first expansion iteration; there each
// thread reads its share of the stamped values, waits (a bounded number of
// polls) until every stamp equals the epoch, and copies them to LDS.  A
// value whose stamp never arrives within the bound is computed by the
// waiting thread itself, so every wave finishes whatever the scheduling.
constexpr int kDBlock = 512, kDWaves = kDBlock / 64;
constexpr int kDTok = 16;                    // tokens per pass (MFMA rows)
#ifndef ARCHEAD_DEC_PREFETCH
#define ARCHEAD_DEC_PREFETCH 3
#endif
constexpr int kDecPD = ARCHEAD_DEC_PREFETCH;  // steps of loads in flight
constexpr int kDecSG = 4;                     // residual groups per step
// Cache policy of the code loads: the default one (the non-temporal hint
// measured 9% slower at 4 tokens on the Qwen-shaped head, where the
// several-token kernel's loads need it).
#ifndef ARCHEAD_DEC_CPOL
#define ARCHEAD_DEC_CPOL 0
#endif
constexpr int kDecCpol = ARCHEAD_DEC_CPOL;

struct DecArgs {
  const uint8_t* codes;
  const uint16_t* rs;
  const uint16_t* rrs;   // row scales of 8-bit residual scale codes (else unused)
  const int8_t* cu;
  const uint16_t* su;
  const int8_t* ca;
  const uint16_t* sa;
  Stage1Ops s1;
  const uint16_t* x;
  int64_t ldx;
  int64_t tok0;          // first token of this pass
  int M;                 // tokens of this pass (1 .. 16)
  int64_t V;
  int d, g, rc, rr;
  int ngrp, kcu, kca;    // residual groups; expansion K-chunks (32 dims) of U_c / A_w
  int cu_row;            // bytes per row of U_c (r_c int8 codes, or ARCHEAD_I5 words)
  int u5;                // U_c codes are ARCHEAD_I5 words
  int64_t n_units;       // ceil(V / 16)
  int64_t n_waves;       // consumer waves (grid-stride over units)
  int n_prod_blocks;     // leading workgroups that compute t
  int xstr;              // LDS: bytes per token row of x
  int tstr;              // LDS: bf16 elements per token row of each part of t
  int off_bias, off_t, off_red;   // LDS byte offsets
  void* out;
  int64_t ldo;
  int out_bf16;
  const void* tgt;
  int tgt64;
  float2* part;          // [tokens, n_part]
  int* part_idx;         // [tokens, n_part] argmax partials, or null
  int64_t n_part;
  float* tgt_logit;
};

// GEN: 0 = the factor codes are read as aligned 8-byte pieces (int8 codes,
// ranks that are multiples of 4); 1 = through fcodes8 (int8 codes, any
// rank); 2 = the same with the core-left codes in ARCHEAD_I5 words.
template <int GW, bool CE, int EK, bool SC8, int GEN>
__global__ __launch_bounds__(kDBlock) __attribute__((amdgpu_waves_per_eu(2)))
void k_dec(DecArgs a) {
  static_assert(GW == 1 || GW == 2 || GW == 4, "code words per lane and group");
  extern __shared__ __align__(16) uint8_t dec_lds[];
  lds_u8* const L = (lds_u8*)dec_lds;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, q = lane >> 4;
  const int M = a.M, d = a.d, g = a.g;
  const int R = a.rc + a.rr;
  const int ngrp = a.ngrp;

  // ---- prologue: x rows of the pass -> LDS, offset biases, zero t padding
  // (every wave of the workgroup calls this once)
  auto prologue = [&]() {
    // x: each thread's 16-byte pieces are requested in batches of 8 before
    // any is stored, so the copy costs one memory latency per batch
    const int x16 = d / 8, nx = M * x16;
    for (int e0 = 0; e0 < nx; e0 += 8 * kDBlock) {
      u32x4_t v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int e0j = e0 + j * kDBlock + tid;
        const int e = e0j < nx ? e0j : nx - 1;   // past the end: a valid piece, not stored
        const int tt = e / x16, u = e - tt * x16;
        v[j] = *reinterpret_cast<const u32x4_t*>(a.x + (a.tok0 + tt) * a.ldx + 8 * u);
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int e = e0 + j * kDBlock + tid;
        const int tt = e / x16, u = e - tt * x16;
        if (e < nx) *reinterpret_cast<__attribute__((address_space(3))) u32x4_t*>(L + tt * a.xstr + 16 * u) = v[j];
      }
    }
    __syncthreads();
    auto* sb = reinterpret_cast<__attribute__((address_space(3))) float*>(L + a.off_bias);
    for (int e = tid; e < ngrp * kDTok; e += kDBlock) {
      const int G = e / kDTok, tt = e % kDTok;
      float s = 0.f;
      if (tt < M) {
        const lds_u8* p = L + tt * a.xstr + 2 * G * g;
        // four pieces per round, requested together
        for (int i = 0; i < g / 8; i += 4) {
          u32x4_t u[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) u[j] = lds_load<u32x4_t>(p + 16 * (i + j < g / 8 ? i + j : i));
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (i + j < g / 8)
              s += bf16_lo(u[j].x) + bf16_hi(u[j].x) + bf16_lo(u[j].y) + bf16_hi(u[j].y) +
                   bf16_lo(u[j].z) + bf16_hi(u[j].z) + bf16_lo(u[j].w) + bf16_hi(u[j].w);
        }
      }
      sb[e] = -float(archead::kInt4Bias) * s;
    }
    auto* st = reinterpret_cast<__attribute__((address_space(3))) uint16_t*>(L + a.off_t);
    for (int e = tid; e < 3 * M * a.tstr; e += kDBlock) st[e] = 0;
    __syncthreads();
  };

  // ---- stage-1 producers: one rank row per wave, all tokens of the pass
  if (int(blockIdx.x) < a.n_prod_blocks) {
    prologue();
    const int k = int(blockIdx.x) * kDWaves + wid;
    if (k < R)
      s1_produce<kDTok>(a.s1, k, M, a.tok0,
                        [&](int tt, int i) { return lds_load<u32x4_t>(L + tt * a.xstr + 2 * i); },
                        lane);
    return;
  }

  // ---- consumers
  const int64_t cw = int64_t(blockIdx.x - a.n_prod_blocks) * kDWaves + wid;
  const int64_t W = a.n_waves;
  const int nu = cw < W ? int((a.n_units - cw + W - 1) / W) : 0;   // units of this wave
  const int kcu = a.kcu, kca = a.kca;      // expansion K-chunks (32 rank dims) of U_c, A_w
  const uint32_t rowbytes = uint32_t(d) / 2;
  const uint32_t kMask = opaque_vgpr(0x000F000Fu);
  const uint32_t kMagic = opaque_vgpr(0x43004300u);
  const int xr = lr < M ? lr : M - 1;                  // token row of this lane's A fragments
  // groups of 64 (GW = 2) are read in pairs, one 128-code block per 16-byte
  // load as for groups of 128 (16 rows x 64 B per load instruction instead
  // of 16 x 32): lane quarter q holds words 4q .. 4q+3 of the pair, so
  // quarters 0-1 hold the first group and 2-3 the second; each group's MFMA
  // chain takes the pair's MFMAs with the other group's lanes zeroed
  constexpr int QW = GW == 2 ? 4 : GW;                 // code words per lane and load
  const lds_u8* const xrow = L + xr * a.xstr + 16 * q * QW;
  const lds_u8* const brow = L + a.off_bias + 16 * q;
  const int tpart = M * a.tstr;                        // bf16 elements per part of t in LDS
  const lds_u8* const trow = L + a.off_t + 2 * (xr * a.tstr);
  // this lane's byte offsets within a unit's rows
  const int voff_c = int(uint32_t(lr) * rowbytes) + q * (4 * QW);        // codes: row lr, quarter q
  constexpr int ESZ = SC8 ? 1 : 2;                                      // bytes per group scale
  const int voff_sc = (lane >> 2) * (ESZ * ngrp) + 16 * (lane & 3);     // scales: row lane/4
  const int voff_u = lr * a.rc + q * (8 * kcu);
  const int voff_a = lr * a.rr + q * (8 * kca);

  CeState<4> ce;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    ce.mx[r] = -INFINITY;
    ce.se[r] = 0.f;
    ce.am[r] = kNoIdx;
    ce.y[r] = -1;
    if (CE && 4 * q + r < M && a.tgt)
      ce.y[r] = a.tgt64 ? reinterpret_cast<const int64_t*>(a.tgt)[a.tok0 + 4 * q + r]
                        : int64_t(reinterpret_cast<const int32_t*>(a.tgt)[a.tok0 + 4 * q + r]);
  }

  // buffer resource over the rows of unit u of an array with `stride` bytes
  // per vocabulary row (rows past V read as zero)
  auto unit_rsrc = [&](const void* base, int64_t u, uint32_t stride) {
    const int64_t v0 = u * 16;
    const uint32_t rows = uint32_t(a.V - v0 < 16 ? a.V - v0 : 16);
    return __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(static_cast<const char*>(base)) + v0 * stride, 0, int(rows * stride),
        kBufferWord3);
  };
  // the same for the U_c / A_w codes, rounded up to whole dwords: a general
  // read takes aligned dwords, and the one holding a unit's last bytes must
  // not come back as zero (any bytes it holds past the buffer are in the
  // same aligned dword, so no further memory is touched, and they belong to
  // dimensions past the rank, paired with zero t)
  auto code_rsrc = [&](const void* base, int64_t u, uint32_t stride) {
    const int64_t v0 = u * 16;
    const int64_t left = a.V - v0;
    const uint32_t rows = uint32_t(left <= 0 ? 0 : (left < 16 ? left : 16));
    return __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(static_cast<const char*>(base)) + (rows ? v0 * stride : 0), 0,
        int((rows * stride + 3) & ~3u), kBufferWord3);
  };
  // The residual scales of a unit (16 rows x d/g, contiguous) arrive as one
  // 16-byte load per lane and 32 fp16 groups (lane l: row l/4, groups
  // 8 (l % 4) .. +7) or 64 8-bit codes (groups 16 (l % 4) .. +15); a lane
  // takes the scales of its own row from the lane holding them with
  // ds_bpermute.
  auto load_scales = [&](int64_t u, u32x4_t (&dst)[2]) {
    const __amdgpu_buffer_rsrc_t r_ = unit_rsrc(a.rs, u, uint32_t(ESZ * ngrp));
    dst[0] = __builtin_amdgcn_raw_buffer_load_b128(r_, voff_sc, 0, 0);
    if (!SC8 && ngrp > 32) dst[1] = __builtin_amdgcn_raw_buffer_load_b128(r_, voff_sc, 64, 0);
  };

  // The head is walked in steps of kDecSG residual groups (one code load
  // per group).
  constexpr int SG = kDecSG;
  const int nsg = ngrp / SG;                     // steps per unit
  constexpr int NB = kDecPD + 1;
  u32x4_t cbuf[NB][SG];
  // load cursor: unit lu (the lk-th of this wave), step lS
  int64_t lu = cw;
  int lk = 0, lS = 0;
  __amdgpu_buffer_rsrc_t lrc = unit_rsrc(a.codes, lu, rowbytes);
  auto load_next = [&](int slot) {
#pragma unroll
    for (int k = 0; k < SG; ++k) {
      const int so = (lS * SG + k) * (g / 2);
      if constexpr (GW == 4) {
        cbuf[slot][k] = __builtin_amdgcn_raw_buffer_load_b128(lrc, voff_c, so, kDecCpol);
      } else if constexpr (GW == 2) {
        if (k % 2 == 0) cbuf[slot][k] = __builtin_amdgcn_raw_buffer_load_b128(lrc, voff_c, so, kDecCpol);
      } else {
        cbuf[slot][k] = u32x4_t{__builtin_amdgcn_raw_buffer_load_b32(lrc, voff_c, so, kDecCpol),
                                0u, 0u, 0u};
      }
    }
    // past the wave's last step the cursor stays there (repeated, unused)
    if (++lS == nsg) {
      if (lk + 1 < nu) {
        lS = 0;
        ++lk;
        lu += W;
        lrc = unit_rsrc(a.codes, lu, rowbytes);
      } else {
        lS = nsg - 1;
      }
    }
  };
  u32x4_t scur[2], snext[2];
  // the first loads of the head go out before the prologue, so the memory
  // works while x, the biases and the t padding are set up
  if (nu > 0) {
    load_scales(cw, scur);
#pragma unroll
    for (int j = 0; j < kDecPD; ++j) load_next(j);
  }
  prologue();

  // t from the producers into LDS, split into three bf16 parts hi = bf16(t),
  // mid = bf16(t - hi), lo = bf16(t - hi - mid) (their sum is t to fp32
  // precision) for the bf16 MFMAs of the expansion.  Every consumer wave
  // takes a share, then a workgroup barrier.  A wave does this when it
  // first needs t, at the end of its first unit (the producers have long
  // finished by then), or at its end if it has no unit.
  bool t_ready = R == 0;
  auto fetch_t = [&]() {
    auto* st = reinterpret_cast<__attribute__((address_space(3))) uint16_t*>(L + a.off_t);
    for (int e = tid; e < M * R; e += kDBlock) {
      const int tt = e / R, k = e - tt * R;
      const float v = s1_value(a.s1, a.tok0, tt, k, [&](int t2, int i) {
        return lds_load<uint32_t>(L + t2 * a.xstr + 2 * i);
      });
      const __bf16 hi = (__bf16)v;
      const float r1 = v - float(hi);
      const __bf16 md = (__bf16)r1;
      const __bf16 lo = (__bf16)(r1 - float(md));
      const int o = tt * a.tstr + (k < a.rc ? k : 32 * kcu + (k - a.rc));
      st[o] = __builtin_bit_cast(uint16_t, hi);
      st[tpart + o] = __builtin_bit_cast(uint16_t, md);
      st[2 * tpart + o] = __builtin_bit_cast(uint16_t, lo);
    }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    t_ready = true;
  };

  if (nu > 0) {
    const int64_t n_it = int64_t(nu) * nsg;
    const int s_issue = nsg > kDecPD ? nsg - kDecPD : 0;   // step that loads the next unit's operands
    int64_t cu_ = cw;   // compute cursor: unit (the ck-th of this wave) and step
    int ck = 0, cS = 0;
    int64_t done_it = 0;
    f32x4_t tot = {0.f, 0.f, 0.f, 0.f};
    // expansion operands of the unit being computed (codes of dims
    // q 8 kc .. +8 kc - 1 of the lane's row, kc K-chunks per part) and its
    // row scales, loaded s_issue steps into the unit
    // EK (2 or 4): the most K-chunks either factor has.  With EK = 2 every
    // load is unconditional (an absent factor's resource has no bytes, and
    // chunks past a factor's rank are read but not used), so no load sits
    // under a branch, which would make the wait-count pass drain the code
    // loads in flight when the unit's operands are requested
    u32x2_t eu[EK], ea[EK];
    uint16_t esu = 0, esa = 0;
    uint16_t ers = 0;   // row scale of 8-bit residual scale codes
    auto load_exp = [&]() {
      const __amdgpu_buffer_rsrc_t ru = code_rsrc(a.cu, cu_, uint32_t(a.cu_row));
      const __amdgpu_buffer_rsrc_t ra = code_rsrc(a.ca, cu_, uint32_t(a.rr));
#pragma unroll
      for (int kc = 0; kc < EK; ++kc) {
        if constexpr (GEN > 0) {
          if (EK == 2 || kc < kcu) eu[kc] = fcodes8<GEN == 2>(ru, lr * a.cu_row, 8 * (q * kcu + kc));
          if (EK == 2 || kc < kca) ea[kc] = fcodes8<false>(ra, lr * a.rr, 8 * (q * kca + kc));
        } else {
          if (EK == 2 || kc < kcu) eu[kc] = __builtin_amdgcn_raw_buffer_load_b64(ru, voff_u, 8 * kc, 0);
          if (EK == 2 || kc < kca) ea[kc] = __builtin_amdgcn_raw_buffer_load_b64(ra, voff_a, 8 * kc, 0);
        }
      }
      if (EK == 2 || kcu) esu = __builtin_amdgcn_raw_buffer_load_b16(unit_rsrc(a.su, cu_, a.rc ? 2u : 0u), 2 * lr, 0, 0);
      if (EK == 2 || kca) esa = __builtin_amdgcn_raw_buffer_load_b16(unit_rsrc(a.sa, cu_, a.rr ? 2u : 0u), 2 * lr, 0, 0);
    };
    auto finish_unit = [&]() {
      if (!t_ready) fetch_t();
      if constexpr (SC8) tot *= f16_to_f32(ers);   // the residual in units of the row scale
      if (kcu + kca > 0) {
        f32x4_t au = {0.f, 0.f, 0.f, 0.f}, aa = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kc = 0; kc < EK; ++kc) {
          if (kc < kcu) {
            const bf16x8_t B = EK == 2 ? int8x8_to_bf16(opaque_vgpr(eu[kc].x), opaque_vgpr(eu[kc].y))
                                       : int8x8_to_bf16(eu[kc].x, eu[kc].y);
            const lds_u8* tp = trow + 2 * (q * 8 * kcu + 8 * kc);
#pragma unroll
            for (int p = 0; p < 3; ++p)
              au = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_load<bf16x8_t>(tp + 2 * p * tpart),
                                                           B, au, 0, 0, 0);
          }
          if (kc < kca) {
            const bf16x8_t B = EK == 2 ? int8x8_to_bf16(opaque_vgpr(ea[kc].x), opaque_vgpr(ea[kc].y))
                                       : int8x8_to_bf16(ea[kc].x, ea[kc].y);
            const lds_u8* tp = trow + 2 * (32 * kcu + q * 8 * kca + 8 * kc);
#pragma unroll
            for (int p = 0; p < 3; ++p)
              aa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lds_load<bf16x8_t>(tp + 2 * p * tpart),
                                                           B, aa, 0, 0, 0);
          }
        }
        tot += f16_to_f32(uint16_t(esu)) * au + f16_to_f32(uint16_t(esa)) * aa;
      }
      const int64_t v = cu_ * 16 + lr;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int tt = 4 * q + r;
        if (tt < M && v < a.V) {
          const float l = tot[r];
          if constexpr (!CE) {
            const int64_t o = (a.tok0 + tt) * a.ldo + v;
            if (a.out_bf16)
              reinterpret_cast<uint16_t*>(a.out)[o] = f32_to_bf16_rne(l);
            else
              reinterpret_cast<float*>(a.out)[o] = l;
          } else {
            if (l > ce.mx[r]) {   // rows come in increasing order per lane
              ce.se[r] = ce.se[r] * fast_exp(ce.mx[r] - l) + 1.f;
              ce.mx[r] = l;
              ce.am[r] = int(v);
            } else {
              ce.se[r] += fast_exp(l - ce.mx[r]);
            }
            if (v == ce.y[r]) a.tgt_logit[a.tok0 + tt] = l;
          }
        }
      }
      tot = f32x4_t{0.f, 0.f, 0.f, 0.f};
    };
    auto body = [&](auto J) {
      constexpr int j = decltype(J)::value;
      load_next((j + kDecPD) % NB);
      asm volatile("" ::: "memory");
      if (cS == s_issue) {
        if (kcu + kca > 0) load_exp();
        if constexpr (SC8)
          ers = __builtin_amdgcn_raw_buffer_load_b16(unit_rsrc(a.rrs, cu_, 2u), 2 * lr, 0, 0);
        if (ck + 1 < nu) load_scales(cu_ + W, snext);
      }
      // scales of this step's groups 4 cS .. 4 cS + 3 of row lr: fp16 in
      // dwords 2 (cS % 2) and 2 (cS % 2) + 1 of lane 4 lr + (cS / 2) % 4's
      // set cS / 8; 8-bit codes in dword cS % 4 of lane 4 lr + cS / 4
      uint32_t s01, s23;
      if constexpr (SC8) {
        const u32x4_t sv = scur[0];
        const int c4 = cS & 3;
        const uint32_t dw = c4 == 0 ? sv[0] : c4 == 1 ? sv[1] : c4 == 2 ? sv[2] : sv[3];
        s01 = uint32_t(__builtin_amdgcn_ds_bpermute(4 * (4 * lr + ((cS >> 2) & 3)), int(dw)));
        s23 = s01;
      } else {
        const u32x4_t sv = cS >= 8 ? scur[1] : scur[0];
        const bool odd = cS & 1;
        const int src = 4 * (4 * lr + ((cS >> 1) & 3));
        s01 = uint32_t(__builtin_amdgcn_ds_bpermute(src, int(odd ? sv[2] : sv[0])));
        s23 = uint32_t(__builtin_amdgcn_ds_bpermute(src, int(odd ? sv[3] : sv[1])));
      }
      f32x4_t acc[SG];
#pragma unroll
      for (int k = 0; k < SG; ++k) acc[k] = lds_load<f32x4_t>(brow + 64 * (cS * SG + k));
      if constexpr (GW == 2) {
        // pair p = groups 2p, 2p+1: the first group's chain sees the codes
        // of quarters 0-1 only (bf16 zeros elsewhere), the second's those of
        // quarters 2-3
        const uint32_t mlo = q < 2 ? 0xffffffffu : 0u;
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) {
#pragma unroll
          for (int p2 = 0; p2 < SG / 2; ++p2) {
            const bf16x8_t A = lds_load<bf16x8_t>(xrow + 2 * (cS * SG + 2 * p2) * g + 16 * kc);
            const u32x4_t B = __builtin_bit_cast(u32x4_t, unpack8(cbuf[j][2 * p2][kc], kMask, kMagic));
            const bf16x8_t B0 = __builtin_bit_cast(bf16x8_t, B & mlo);
            const bf16x8_t B1 = __builtin_bit_cast(bf16x8_t, B & ~mlo);
            acc[2 * p2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B0, acc[2 * p2], 0, 0, 0);
            acc[2 * p2 + 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B1, acc[2 * p2 + 1], 0, 0, 0);
          }
        }
      } else {
#pragma unroll
        for (int kc = 0; kc < GW; ++kc) {
#pragma unroll
          for (int k = 0; k < SG; ++k) {
            const bf16x8_t A = lds_load<bf16x8_t>(xrow + 2 * (cS * SG + k) * g + 16 * kc);
            acc[k] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                A, unpack8(cbuf[j][k][kc], kMask, kMagic), acc[k], 0, 0, 0);
          }
        }
      }
#pragma unroll
      for (int k = 0; k < SG; ++k) {
        if constexpr (SC8) {
          tot += float((s01 >> (8 * k)) & 0xffu) * acc[k];
        } else {
          const uint32_t sw = k < 2 ? s01 : s23;
          tot += f16_to_f32(uint16_t(k & 1 ? sw >> 16 : sw)) * acc[k];
        }
      }
      if (++cS == nsg) {
        finish_unit();
        cS = 0;
        cu_ += W;
        ++ck;
        scur[0] = snext[0];
        scur[1] = snext[1];
      }
      return ++done_it == n_it;
    };
    while (!unroll_until<0, NB>(body)) {
    }
  }
  if (!t_ready) fetch_t();

  if constexpr (CE) {
    // per token: merge the 16 rows' states of each quarter, then the waves
    float2* red = reinterpret_cast<float2*>(dec_lds + a.off_red);   // [kDWaves][kDTok]
    int* redi = reinterpret_cast<int*>(red + kDWaves * kDTok);       // [kDWaves][kDTok]
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float m = row16_max(ce.mx[r]);
      float se = m == -INFINITY ? 0.f : ce.se[r] * fast_exp(ce.mx[r] - m);
      se = row16_sum(se);
      const int ai = row16_min_i(ce.mx[r] == m ? ce.am[r] : kNoIdx);
      if (lr == 0) {
        red[wid * kDTok + 4 * q + r] = make_float2(m, se);
        redi[wid * kDTok + 4 * q + r] = ai;
      }
    }
    __syncthreads();
    if (tid < M) {
      float m = red[tid].x, s = red[tid].y;
      for (int w = 1; w < kDWaves; ++w) lse_merge(m, s, red[w * kDTok + tid].x, red[w * kDTok + tid].y);
      const int64_t o = (a.tok0 + tid) * a.n_part + (blockIdx.x - a.n_prod_blocks);
      a.part[o] = make_float2(m, s);
      if (a.part_idx) {
        int ai = kNoIdx;
        for (int w = 0; w < kDWaves; ++w)
          if (red[w * kDTok + tid].x == m) ai = min(ai, redi[w * kDTok + tid]);
        a.part_idx[o] = ai;
      }
    }
  }
}

}  // namespace
