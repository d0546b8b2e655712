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

#include <algorithm>
#include <atomic>
#include <chrono>
#include <type_traits>
#include <stdint.h>
#include <string.h>

#include "archead.h"
#include "internal.h"

namespace {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

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
// four bytes (integers 0..255, exact in fp16) as four fp16, low byte first
__device__ __forceinline__ u32x2_t u8x4_to_f16x4(uint32_t w) {
  auto h = [](uint32_t b) {
    return uint32_t(__builtin_bit_cast(uint16_t, _Float16(float(b & 0xffu))));
  };
  return u32x2_t{h(w) | (h(w >> 8) << 16), h(w >> 16) | (h(w >> 24) << 16)};
}
__device__ __forceinline__ float bf16_lo(uint32_t p) { return __uint_as_float(p << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t p) { return __uint_as_float(p & 0xffff0000u); }

// (x & m) | o, selected as one v_and_or_b32.  With literal m and o the
// compiler would split it into v_and + v_or (gfx9 VOP3 takes no literal), so
// callers pass m and o through opaque_vgpr(), which hides their values and
// keeps them in registers.  Plain C rather than inline asm: the hazard
// recognizer does not see into inline asm, and a VALU write into a register
// an in-flight MFMA still reads needs wait states it would then not insert.
__device__ __forceinline__ uint32_t opaque_vgpr(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}
// A kernel argument as an opaque wave-uniform register value.  A per-lane
// select between two fields of the argument block would otherwise become a
// load through a per-lane address (a vector-memory load whose wait also
// drains every load in flight); between two registers it stays a select.
template <typename T>
__device__ __forceinline__ T opaque_sgpr(T v) {
  asm volatile("" : "+s"(v));
  return v;
}
__device__ __forceinline__ uint32_t and_or(uint32_t x, uint32_t m, uint32_t o) {
  return (x & m) | o;
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

// ------------------------------------------------ stage 1 inside the launch
// The decode GEMV, the MFMA decode kernel and the several-token kernel
// compute t = x V_c^T, x B_w^T in the same launch as the head stream: the first workgroups of the grid ("producers") take one rank
// row per wave and publish each value t[m][k] together with the call's
// epoch in one 64-bit store (agent scope, so the value and its stamp become
// visible together on every XCD).  The other waves need t only at the end of
// their first vocabulary step; they read the stamped values, poll a bounded
// number of times until every stamp equals the epoch, and compute any value
// whose stamp has not arrived by then themselves, so every wave finishes
// whatever the scheduling of the producers.
struct Stage1Ops {
  const int8_t* cv;      // V_c codes [r_c, d], group scales [r_c, d / gv]
  const uint16_t* sv;
  const int8_t* cb;      // B_w codes [r_r, d], group scales [r_r, d / gb]
  const uint16_t* sb;
  int gv, gb, rc, rr, d;
  unsigned long long* tst;   // [tokens][r_c + r_r]: float bits | epoch << 32
  uint32_t epoch;
  int spin_limit;            // polls before the fallback
};

__device__ __forceinline__ unsigned long long load_stamped(const unsigned long long* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Producer: t[tok0 + tt][k] for tt < M of rank row k (V_c rows first, then
// B_w), one wave; x8(tt, i) gives the 8 bf16 values x[tt][i .. i + 7].
// s * c is exact in fp32 (11 x 8 significant bits); fp32 accumulation.
template <int TOKMAX, typename X8>
__device__ __forceinline__ void s1_produce(const Stage1Ops& s, int k, int M, int64_t tok0,
                                           X8 x8, int lane) {
  const int d = s.d, R = s.rc + s.rr;
  const bool core = k < s.rc;
  const int8_t* crow = core ? s.cv + int64_t(k) * d : s.cb + int64_t(k - s.rc) * d;
  const int grp = core ? s.gv : s.gb;
  const uint16_t* srow =
      core ? s.sv + int64_t(k) * (d / s.gv) : s.sb + int64_t(k - s.rc) * (d / s.gb);
  float acc[TOKMAX];
#pragma unroll
  for (int tt = 0; tt < TOKMAX; ++tt) acc[tt] = 0.f;
  // 8 pieces of 8 codes per lane at a time, all loads issued before the
  // arithmetic (the head stream keeps the memory busy, so each round trip is
  // long)
  constexpr int kPieces = 8;
  for (int base = lane * 8; base < d; base += 512 * kPieces) {
    uint2 cw[kPieces];
    uint16_t sw[kPieces];
#pragma unroll
    for (int p = 0; p < kPieces; ++p) {
      const int i = base + 512 * p;
      const int ic = i < d ? i : base;
      cw[p] = *reinterpret_cast<const uint2*>(crow + ic);
      sw[p] = srow[ic / grp];
    }
#pragma unroll
    for (int p = 0; p < kPieces; ++p) {
      const int i = base + 512 * p;
      if (i < d) {
        const float sc = f16_to_f32(sw[p]);
        float w[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          w[j] = float(int8_t(cw[p].x >> (8 * j))) * sc;
          w[4 + j] = float(int8_t(cw[p].y >> (8 * j))) * sc;
        }
#pragma unroll
        for (int tt = 0; tt < TOKMAX; ++tt) {
          if (tt < M) {
            const u32x4_t xv = x8(tt, i);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              acc[tt] = fmaf(bf16_lo(xv[j]), w[2 * j], acc[tt]);
              acc[tt] = fmaf(bf16_hi(xv[j]), w[2 * j + 1], acc[tt]);
            }
          }
        }
      }
    }
  }
#pragma unroll
  for (int tt = 0; tt < TOKMAX; ++tt) {
    if (tt < M) {
      const float v = seg_sum<64>(acc[tt]);
      if (lane == tt) {
        const unsigned long long word =
            (static_cast<unsigned long long>(s.epoch) << 32) | __float_as_uint(v);
        __hip_atomic_store(s.tst + (tok0 + tt) * R + k, word, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
}

// Consumer: t[tok0 + tt][k], from its stamped word once the stamp equals the
// epoch, else (after spin_limit polls) computed here by one thread in
// element order; x2(tt, i) gives the bf16 pair x[tt][i], x[tt][i + 1].
template <typename X2>
__device__ float s1_value(const Stage1Ops& s, int64_t tok0, int tt, int k, X2 x2) {
  const int R = s.rc + s.rr;
  const unsigned long long* p = s.tst + (tok0 + tt) * R + k;
  unsigned long long w = load_stamped(p);
  for (int it = 0; uint32_t(w >> 32) != s.epoch && it < s.spin_limit; ++it) {
    __builtin_amdgcn_s_sleep(2);
    w = load_stamped(p);
  }
  if (uint32_t(w >> 32) == s.epoch) return __uint_as_float(uint32_t(w));
  const bool core = k < s.rc;
  const int8_t* crow = core ? s.cv + int64_t(k) * s.d : s.cb + int64_t(k - s.rc) * s.d;
  const int grp = core ? s.gv : s.gb;
  const uint16_t* srow =
      core ? s.sv + int64_t(k) * (s.d / s.gv) : s.sb + int64_t(k - s.rc) * (s.d / s.gb);
  float acc = 0.f;
  for (int i = 0; i < s.d; i += 2) {
    const float sc = f16_to_f32(srow[i / grp]);
    const uint32_t xp = x2(tt, i);
    acc = fmaf(bf16_lo(xp), float(crow[i]) * sc, acc);
    acc = fmaf(bf16_hi(xp), float(crow[i + 1]) * sc, acc);
  }
  return acc;
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
  uint16_t rsc[RB];     // fp16 row scale of 8-bit residual scale codes (unused otherwise)
  uint16_t s[RB][KD];   // fp16 bit pattern of the row scale (kept 16-bit: no extension op right after the load)
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

// Per-lane softmax state of the fused CE epilogue.
template <int TOK>
struct CeState {
  float mx[TOK], se[TOK];
  int am[TOK];      // smallest vocabulary index attaining mx so far
  int64_t y[TOK];
};

// "no index yet" for the argmax partials: larger than any vocabulary index
constexpr int kNoIdx = 0x7fffffff;

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
template <int TOK, int LPR, bool CE, bool SC8>
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
  uint16_t* sx = reinterpret_cast<uint16_t*>(smem);          // [TOK][d]
  float* sxb = reinterpret_cast<float*>(sx + TOK * d);        // [TOK][C]
  const int wid = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  float* st = sxb + TOK * C + wid * TOK * R;                  // this wave's t [TOK][R]
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
    for (int i = threadIdx.x; i < TOK * x8n; i += kBlock) {
      const int tt = i / x8n, u = i - tt * x8n;
      reinterpret_cast<uint4*>(sx)[(tt * 4 + (u & 3)) * C + (u >> 2)] =
          *reinterpret_cast<const uint4*>(a.x + (a.tok0 + tt) * a.ldx + u * 8);
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
    for (int e = lane; e < TOK * R; e += 64) {
      const int tt = e / R;
      st[e] = s1_value(a.s1, a.tok0, tt, e - tt * R, x2);
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
    const int rc4 = a.rc / 4, R4 = R / 4;
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
    const int64_t cu_st = opaque_sgpr(a.cu_stride), ca_st = opaque_sgpr(a.ca_stride);
    const int64_t su_st = opaque_sgpr(a.su_stride), sa_st = opaque_sgpr(a.sa_stride);
    auto load_exp = [&](int64_t stp, ExpOps<RB, KD>& e) {
      const int64_t v0 = stp * WR + seg;
#pragma unroll
      for (int kd = 0; kd < KD; ++kd) {
        int q = sl + kd * LPR;
        q = q < R4 ? q : 0;
        const bool isu = q < rc4;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const int64_t v = v0 + rb * SEG;
          const int8_t* cb = isu ? a.cu + 4 * q + v * cu_st : a.ca + 4 * (q - rc4) + v * ca_st;
          const uint16_t* sp = isu ? a.su + v * su_st : a.sa + v * sa_st;
          e.c[rb][kd] = *reinterpret_cast<const uint32_t*>(cb);
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
        apply_expansion<TOK, RB, KD, LPR>(acc, e, st, R, sl);
        load_exp(more ? nstep : cstep, e);
        gemv_epilogue<TOK, LPR, RB, CE, false>(acc, a, cstep * WR, uint32_t(WR - 1), seg, sl,
                                               lane, my_row, writer, st, ce);
      }
      cstep = nstep;
      cit = nit;
      done = !more;
    };
    while (gw < full_steps) {
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
    gemv_epilogue<TOK, LPR, RB, CE, true>(acc, a, row0, lim, seg, sl, lane, my_row, writer, st,
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
}

// ------------------------------------------------------------ many tokens: MFMA
// Tiled bf16 MFMA path for many tokens (needs g % 64 == 0).  A workgroup owns
// a kTM x kTN tile (tokens x vocabulary rows); its eight waves own 128 x 64
// blocks (2 along the tokens, 4 along the vocabulary), each an 8 x 4 grid of
// 16x16 MFMA tiles (v_mfma_f32_16x16x32_bf16: A lane l holds row l%16 and 8
// k-slots of quarter l/16; B likewise by column; D lane l holds rows
// 4 (l/16) .. +3 of column l%16).  The K loop runs in stages of kKS elements
// that direct global-to-LDS buffer loads bring into a ring of kRing LDS
// stages, two stages ahead of the compute, with no register staging.  Within
// a stage lane quarter q takes code dwords 2q, 2q+1 (one per MFMA K-chunk)
// and the x chunks with the same indices, so its codes are one 8-byte read.
// Token rows and vocabulary rows are XOR-swizzled in 16-byte units so
// fragment reads are bank-conflict free.
//
// Codes are unpacked per wave to bf16 (136 + c) (exact).  The accumulator is
// kept in units of the current scale slot's scale: at the start of slot k it
// becomes acc * (s'_{k-1} / s'_k) + bias_k, after which the MFMAs add the
// slot's terms, so at the end s'_last * acc is the logit.  Slots are the
// residual groups (bias -136 * (sum of x over the group), the MFMAs adding
// sum (136 + c) x), then the rank-r expansion's core part (scale s_U) and
// correction part (s_A).  s' is the scale with zero replaced by kZeroScale,
// which pushes a zero-scale slot's contribution below fp32 resolution of the
// result.  The expansion parts run as extra stages with the same geometry,
// 16 rank dimensions per stage: the "x" rows hold t split into three bf16
// parts (hi = bf16(t), mid = bf16(t - hi), lo = bf16(t - hi - mid); their sum
// is t to fp32 precision) as [hi | mid | lo | 0], the "code" rows the int8
// factor codes (exact in bf16) twice, [c | c], so MFMA K-chunk 0 adds
// (hi + mid) c and K-chunk 1 adds lo c.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) uint8_t lds_u8;

constexpr int kTM = 256, kTN = 256;          // tile: tokens x vocabulary rows
constexpr int kMBlock = 512, kMWaves = 8;    // 2 x 4 waves of 128 x 64
constexpr int kKS = 64;                      // K elements per stage
constexpr int kRing = 3;                     // LDS stages (two loads in flight)
constexpr int kRasterGM = 2;                 // token tiles per raster group
constexpr float kZeroScale = 0x1p-60f;       // stand-in for a zero scale
constexpr int kExpDims = 16;                 // rank dimensions per expansion stage

struct MGeom {
  static constexpr int XBYTES = kTM * kKS * 2;        // x [kTM][kKS] bf16
  static constexpr int CBYTES = kTN * kKS / 2;        // codes [kTN][kKS/2]
  static constexpr int RAT = XBYTES + CBYTES;         // fp32 [kTN] scale ratios
  static constexpr int BIAS = RAT + kTN * 4;          // fp32 [kTM] slot biases
  static constexpr int STAGE = BIAS + kTM * 4;
  static constexpr int NX = XBYTES / 1024 / kMWaves;  // x loads per wave and stage
  static constexpr int NL = NX + 2;                   // loads per wave and stage
  static constexpr int LDS = kRing * STAGE;
  static_assert(CBYTES / 1024 == kMWaves, "one code load per wave");
  static_assert(LDS <= 160 * 1024, "LDS budget");
};

// 16-byte unit swizzles; only the low four bits of the row matter, so every
// lane's swizzle is fixed for all its fragments
__device__ __forceinline__ int swz_x(int r) { return ((r & 15) ^ ((r & 15) >> 3)) & 7; }
__device__ __forceinline__ int swz_c(int c) { return (c >> 2) & 1; }

__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, lds_u8* dst, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(
      r, reinterpret_cast<__attribute__((address_space(3))) void*>(dst), 16, voff, 0, 0, 0);
}
__device__ __forceinline__ void dma4(__amdgpu_buffer_rsrc_t r, lds_u8* dst, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(
      r, reinterpret_cast<__attribute__((address_space(3))) void*>(dst), 4, voff, 0, 0, 0);
}

// Wait until at most N of this wave's vector-memory loads are in flight and
// its LDS reads are done, then meet the other waves.  The memory clobber
// keeps LDS accesses on their side of it.
template <int N>
__device__ __forceinline__ void wait_loads_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

template <typename T>
__device__ __forceinline__ T lds_load(const lds_u8* p) {
  return *reinterpret_cast<const __attribute__((address_space(3))) T*>(p);
}

__device__ __forceinline__ bf16x8_t unpack8(uint32_t q, uint32_t kMask, uint32_t kMagic) {
  uint32_t p[4];
  p[0] = int4_pair<0>(q, kMask, kMagic);
  p[1] = int4_pair<1>(q, kMask, kMagic);
  p[2] = int4_pair<2>(q, kMask, kMagic);
  p[3] = int4_pair<3>(q, kMask, kMagic);
  return __builtin_bit_cast(bf16x8_t, p);
}

// max / sum over the 16 lanes of a row (DPP lane swaps within the row:
// quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror, row_mirror)
template <int CTRL>
__device__ __forceinline__ float dpp_swap(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_swap<0xB1>(v));
  v = fmaxf(v, dpp_swap<0x4E>(v));
  v = fmaxf(v, dpp_swap<0x141>(v));
  return fmaxf(v, dpp_swap<0x140>(v));
}
__device__ __forceinline__ int row16_min_i(int v) {
  v = min(v, __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false));
  v = min(v, __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false));
  v = min(v, __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false));
  return min(v, __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false));
}
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_swap<0xB1>(v);
  v += dpp_swap<0x4E>(v);
  v += dpp_swap<0x141>(v);
  return v + dpp_swap<0x140>(v);
}

// eight int8 codes (little-endian in two dwords) as bf16 (exact)
__device__ __forceinline__ bf16x8_t int8x8_to_bf16(uint32_t w0, uint32_t w1) {
  uint32_t p[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t w = j < 2 ? w0 : w1;
    const int sh = 16 * (j & 1);
    const float lo = float(int8_t(w >> sh)), hi = float(int8_t(w >> (sh + 8)));
    p[j] = __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
  }
  return __builtin_bit_cast(bf16x8_t, p);
}

struct MfmaArgs {
  const uint8_t* codes;
  const uint16_t* x;
  int64_t ldx;
  const uint16_t* tsplit;  // [M][nch][4][16] bf16: t hi, mid, lo, 0 per 16 rank dimensions
  const int8_t* ucodes;    // [V][nch][2][16] int8: U_c then A_w codes (each padded), twice
  const float* gbias;      // [n_mt][nslot][kTM] slot biases
  const float* ratio;      // [n_vt][nslot][kTN]: s'_{k-1} / s'_k (0 for k = 0)
  const float* fin;        // [n_vt][kTN]: s' of the last slot
  int64_t M, V;
  int d, g, nslot, nch, nch_u;
  int64_t n_mt, n_vt, n_tiles, tiles_per_xcd;
  void* out;
  int64_t ldo;
  int out_bf16;
  const void* tgt;
  int tgt64;
  float2* part;            // [M, n_vt]
  int* part_idx;           // [M, n_vt] argmax partials, or null
  float* tgt_logit;        // [M]
};

template <bool CE>
__global__ __launch_bounds__(kMBlock) void k_mfma(MfmaArgs a) {
  using G = MGeom;
  extern __shared__ __align__(16) uint8_t mfma_lds[];
  lds_u8* const L = (lds_u8*)mfma_lds;

  // tile: workgroups are dealt to the 8 XCDs round-robin, so XCD x runs
  // blocks x, x+8, ...; it gets the contiguous run [x T, (x+1) T) of the tile
  // order, which walks groups of kRasterGM token tiles across the vocabulary
  // (token tile fastest): the tiles one XCD runs at once share a few token
  // tiles and a few vocabulary tiles in its L2
  const int64_t b = blockIdx.x;
  const int64_t lin = (b & 7) * a.tiles_per_xcd + (b >> 3);
  if (lin >= a.n_tiles) return;
  const int64_t gsz = int64_t(kRasterGM) * a.n_vt;
  const int64_t rg = lin / gsz, first = rg * kRasterGM;
  const int64_t gm = a.n_mt - first < kRasterGM ? a.n_mt - first : kRasterGM;
  const int64_t within = lin - rg * gsz;
  const int64_t mt = first + within % gm, vt = within / gm;
  const int64_t m0 = mt * kTM, v0 = vt * kTN;
  const int rows = int(a.M - m0 < kTM ? a.M - m0 : kTM);
  const int cols = int(a.V - v0 < kTN ? a.V - v0 : kTN);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 2, wn = wid & 3;
  const int lr = lane & 15, q = lane >> 4;
  const uint32_t kMask = opaque_vgpr(0x000F000Fu);
  const uint32_t kMagic = opaque_vgpr(0x43004300u);
  const int ngrp = a.d / a.g;
  const uint32_t rowbytes = uint32_t(a.d) / 2;
  const uint32_t ldx2 = uint32_t(a.ldx) * 2;
  const uint32_t trow = uint32_t(a.nch) * 128, urow = uint32_t(a.nch) * 32;

  // buffer resources over exactly the bytes this tile may touch (loads past
  // them return zero instead of reading other memory)
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.x + m0 * a.ldx), 0, int((rows - 1) * ldx2 + uint32_t(a.d) * 2),
      kBufferWord3);
  const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(a.codes + v0 * int64_t(rowbytes)), 0, int(uint32_t(cols) * rowbytes),
      kBufferWord3);
  const __amdgpu_buffer_rsrc_t rt = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.tsplit + m0 * int64_t(a.nch) * 64), 0, int(uint32_t(rows) * trow),
      kBufferWord3);
  const __amdgpu_buffer_rsrc_t ru = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int8_t*>(a.ucodes + v0 * int64_t(urow)), 0, int(uint32_t(cols) * urow),
      kBufferWord3);
  // auxiliary load of this wave: scale ratios (waves 0-3, 64 columns each)
  // or slot biases (waves 4-7, 64 token rows each)
  const bool arat = wid < 4;
  const __amdgpu_buffer_rsrc_t raux =
      arat ? __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.ratio + vt * a.nslot * kTN),
                                               0, a.nslot * kTN * 4, kBufferWord3)
           : __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.gbias + mt * a.nslot * kTM),
                                               0, a.nslot * kTM * 4, kBufferWord3);

  // per-lane load offsets (row and swizzled 16-byte unit) of the residual
  // stages; the expansion stages use the same units with their own row
  // strides; the stage's k offset is added per stage
  auto xunit = [&](int i, uint32_t stride) {
    const int off = (wid * G::NX + i) * 1024 + 16 * lane;
    const int r = off / (2 * kKS), p = (off % (2 * kKS)) / 16;
    return uint32_t(r < rows ? r : rows - 1) * stride + 16u * uint32_t(p ^ swz_x(r));
  };
  auto cunit = [&](uint32_t stride) {
    const int off = wid * 1024 + 16 * lane;
    const int c = off / (kKS / 2), p = (off % (kKS / 2)) / 16;
    return uint32_t(c < cols ? c : cols - 1) * stride + 16u * uint32_t(p ^ swz_c(c));
  };
  uint32_t xo[G::NX];
#pragma unroll
  for (int i = 0; i < G::NX; ++i) xo[i] = xunit(i, ldx2);
  const uint32_t co = cunit(rowbytes);
  uint32_t ao;
  int adst;
  if (arat) {
    ao = uint32_t(wid * 64 + lane) * 4;
    adst = G::RAT + wid * 256;
  } else {
    const int r = (wid - 4) * 64 + lane;
    ao = uint32_t(r < rows ? r : rows - 1) * 4;
    adst = G::BIAS + (wid - 4) * 256;
  }

  const int nst = a.d / kKS, spg = a.g / kKS, ntot = nst + a.nch;
  const int slot_u = ngrp, slot_a = ngrp + (a.nch_u > 0 ? 1 : 0);
  auto slot_of = [&](int s) {
    return s < nst ? s / spg : (s - nst < a.nch_u ? slot_u : slot_a);
  };
  // load PART (0 .. NL-1) of this wave's share of stage s into ring slot buf
  auto issue_part = [&](int s, int buf, int part) {
    lds_u8* base = L + buf * G::STAGE;
    if (part < G::NX) {
      if (s < nst) dma16(rx, base + (wid * G::NX + part) * 1024, xo[part] + uint32_t(s) * (kKS * 2));
      else dma16(rt, base + (wid * G::NX + part) * 1024, xunit(part, trow) + uint32_t(s - nst) * 128);
    } else if (part == G::NX) {
      if (s < nst) dma16(rc, base + G::XBYTES + wid * 1024, co + uint32_t(s) * (kKS / 2));
      else dma16(ru, base + G::XBYTES + wid * 1024, cunit(urow) + uint32_t(s - nst) * 32);
    } else {
      dma4(raux, base + adst, ao + uint32_t(slot_of(s)) * 1024u);
    }
  };
  auto issue = [&](int s, int buf) {
#pragma unroll
    for (int part = 0; part < G::NL; ++part) issue_part(s, buf, part);
  };
  // the same for a stage known to be a residual / an expansion stage
  auto issue_main = [&](int s, int buf, int part) {
    lds_u8* base = L + buf * G::STAGE;
    if (part < G::NX) dma16(rx, base + (wid * G::NX + part) * 1024, xo[part] + uint32_t(s) * (kKS * 2));
    else if (part == G::NX) dma16(rc, base + G::XBYTES + wid * 1024, co + uint32_t(s) * (kKS / 2));
    else dma4(raux, base + adst, ao + uint32_t(s / spg) * 1024u);
  };
  auto issue_exp = [&](int s, int buf, int part) {
    lds_u8* base = L + buf * G::STAGE;
    if (part < G::NX) dma16(rt, base + (wid * G::NX + part) * 1024, xunit(part, trow) + uint32_t(s - nst) * 128);
    else if (part == G::NX) dma16(ru, base + G::XBYTES + wid * 1024, cunit(urow) + uint32_t(s - nst) * 32);
    else dma4(raux, base + adst, ao + uint32_t(slot_of(s)) * 1024u);
  };

  // fragment offsets within a stage: residual stages take x chunks 2q + kc,
  // expansion stages chunk 4 kc + q ([hi | mid] for kc = 0, [lo | 0] for
  // kc = 1), matched by code dimensions 8 (q % 2) .. +7 of [c | c]
  const uint32_t arow = uint32_t(128 * wm + lr) * (2 * kKS);
  uint32_t aoff[2];
#pragma unroll
  for (int kc = 0; kc < 2; ++kc) aoff[kc] = arow + 16u * uint32_t((2 * q + kc) ^ swz_x(lr));
  const uint32_t boff =
      G::XBYTES + uint32_t(64 * wn + lr) * 32 + 16u * uint32_t((q >> 1) ^ swz_c(lr)) + 8u * (q & 1);

  f32x4_t acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // final scales and (CE) the targets of the tile's rows, loaded before the
  // stage loads so they have arrived by the epilogue
  float fin[4];
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) fin[ni] = a.fin[vt * kTN + 64 * wn + 16 * ni + lr];
  int64_t y_row = -1;
  if (CE && tid < rows && a.tgt)
    y_row = a.tgt64 ? reinterpret_cast<const int64_t*>(a.tgt)[m0 + tid]
                    : int64_t(reinterpret_cast<const int32_t*>(a.tgt)[m0 + tid]);
  issue(0, 0);
  if (ntot > 1) issue(1, 1);
  // The loads of stage s + 2 are issued one part at a time between the
  // MFMAs of stage s's first K-chunk, so the waves' vector-memory traffic
  // does not queue up in one burst after the barrier.
  int buf = 0;   // ring slot of the next stage to compute
  auto next_stage = [&](int s) {
    if (s + 1 < ntot) wait_loads_barrier<G::NL>();
    else wait_loads_barrier<0>();
    const lds_u8* base = L + buf * G::STAGE;
    buf = buf == 2 ? 0 : buf + 1;
    return base;
  };
  static_assert(G::NL <= 8, "one load per MFMA row block of the first K-chunk");
  // slot start: rescale to the slot's scale and add its bias
  auto rescale = [&](const lds_u8* base) {
    float rat[4];
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) rat[ni] = lds_load<float>(base + G::RAT + (64 * wn + 16 * ni + lr) * 4);
#pragma unroll
    for (int mi = 0; mi < 8; ++mi) {
      const f32x4_t bias = lds_load<f32x4_t>(base + G::BIAS + (128 * wm + 16 * mi + 4 * q) * 4);
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = acc[mi][ni] * rat[ni] + bias;
    }
  };

  // Stage bodies; ISSUE says how the loads of stage s + 2 are issued:
  // 0 none, 1 residual source, 2 expansion source, 3 either (checked).
  int sg = 0;   // stage index within its scale group
  auto main_stage = [&](int s, auto issue_kind) {
    constexpr int ISSUE = decltype(issue_kind)::value;
    const lds_u8* base = next_stage(s);
    const int nb = buf == 2 ? 0 : buf + 1;   // ring slot of stage s + 2
    u32x2_t braw[4];
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) braw[ni] = lds_load<u32x2_t>(base + boff + ni * 16 * (kKS / 2));
    bf16x8_t A[8];
#pragma unroll
    for (int mi = 0; mi < 8; ++mi) A[mi] = lds_load<bf16x8_t>(base + aoff[0] + mi * 32 * kKS);
    if (sg == 0) rescale(base);
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      bf16x8_t B[4];
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) B[ni] = unpack8(braw[ni][kc], kMask, kMagic);
#pragma unroll
      for (int mi = 0; mi < 8; ++mi) {
        const bf16x8_t Am = A[mi];
        if (kc == 0) A[mi] = lds_load<bf16x8_t>(base + aoff[1] + mi * 32 * kKS);
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Am, B[ni], acc[mi][ni], 0, 0, 0);
        if (kc == 0 && mi < G::NL) {
          if constexpr (ISSUE == 1) issue_main(s + 2, nb, mi);
          if constexpr (ISSUE == 3) if (s + 2 < ntot) issue_part(s + 2, nb, mi);
        }
      }
    }
    sg = sg == spg - 1 ? 0 : sg + 1;
  };
  auto exp_stage = [&](int s, auto issue_kind) {
    constexpr int ISSUE = decltype(issue_kind)::value;
    const lds_u8* base = next_stage(s);
    const int nb = buf == 2 ? 0 : buf + 1;
    u32x2_t braw[4];
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) braw[ni] = lds_load<u32x2_t>(base + boff + ni * 16 * (kKS / 2));
    if (s == nst || s == nst + a.nch_u) rescale(base);
    bf16x8_t B[4];
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) B[ni] = int8x8_to_bf16(braw[ni].x, braw[ni].y);
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      const uint32_t eoff = arow + 16u * uint32_t((4 * kc + q) ^ swz_x(lr));
#pragma unroll
      for (int mi = 0; mi < 8; ++mi) {
        const bf16x8_t A = lds_load<bf16x8_t>(base + eoff + mi * 32 * kKS);
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B[ni], acc[mi][ni], 0, 0, 0);
        if (kc == 0 && mi < G::NL) {
          if constexpr (ISSUE == 2) issue_exp(s + 2, nb, mi);
          if constexpr (ISSUE == 3) if (s + 2 < ntot) issue_part(s + 2, nb, mi);
        }
      }
    }
  };
  using kNone = std::integral_constant<int, 0>;
  using kMain = std::integral_constant<int, 1>;
  using kExp = std::integral_constant<int, 2>;
  using kAny = std::integral_constant<int, 3>;
  int s = 0;
#pragma unroll 1
  for (; s + 2 < nst; ++s) main_stage(s, kMain{});
#pragma unroll 1
  for (; s < nst; ++s) main_stage(s, kAny{});
#pragma unroll 1
  for (; s + 2 < ntot; ++s) exp_stage(s, kExp{});
#pragma unroll 1
  for (; s < ntot; ++s) exp_stage(s, kNone{});
#pragma unroll
  for (int ni = 0; ni < 4; ++ni)
#pragma unroll
    for (int mi = 0; mi < 8; ++mi) acc[mi][ni] *= fin[ni];

  // ---- epilogue
  if constexpr (!CE) {
#pragma unroll
    for (int mi = 0; mi < 8; ++mi)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = 128 * wm + 16 * mi + 4 * q + i;
        if (row >= rows) continue;
        const int64_t m = m0 + row;
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          const int col = 64 * wn + 16 * ni + lr;
          if (col >= cols) continue;
          const float l = acc[mi][ni][i];
          if (a.out_bf16)
            reinterpret_cast<uint16_t*>(a.out)[m * a.ldo + v0 + col] = f32_to_bf16_rne(l);
          else
            reinterpret_cast<float*>(a.out)[m * a.ldo + v0 + col] = l;
        }
      }
  } else {
    // per token row: (max, sum exp) over this tile's valid columns; the 16
    // lanes of a quarter-wave share rows, the four waves along the
    // vocabulary are merged through LDS in a fixed order.  Targets are
    // staged in LDS as tile-local columns (-1: not in this tile).
    float2* sred = reinterpret_cast<float2*>(mfma_lds);               // [4][kTM]
    int* sy = reinterpret_cast<int*>(mfma_lds + 4 * kTM * sizeof(float2));   // [kTM]
    int* sidx = sy + kTM;                                                // [4][kTM] argmax
    __syncthreads();
    if (tid < kTM) sy[tid] = y_row >= v0 && y_row < v0 + cols ? int(y_row - v0) : -1;
    __syncthreads();
    // IDX: also the smallest tile column at each row's maximum (argmax
    // partials); compiled apart so the CE-only pass pays nothing for it
    auto rows_pass = [&](auto IDX) {
      constexpr bool kIdx = decltype(IDX)::value;
#pragma unroll
      for (int mi = 0; mi < 8; ++mi)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = 128 * wm + 16 * mi + 4 * q + i;
          const int yl = sy[row];
          float mx = -INFINITY;
#pragma unroll
          for (int ni = 0; ni < 4; ++ni)
            if (64 * wn + 16 * ni + lr < cols) mx = fmaxf(mx, acc[mi][ni][i]);
          mx = row16_max(mx);
          float se = 0.f;
          int ai = kNoIdx;
#pragma unroll
          for (int ni = 0; ni < 4; ++ni) {
            const int col = 64 * wn + 16 * ni + lr;
            if (col < cols) {
              se += fast_exp(acc[mi][ni][i] - mx);
              if (col == yl) a.tgt_logit[m0 + row] = acc[mi][ni][i];
              if (kIdx && acc[mi][ni][i] == mx) ai = min(ai, col);
            }
          }
          se = row16_sum(se);
          if constexpr (kIdx) ai = row16_min_i(ai);
          if (lr == 0) {
            sred[wn * kTM + row] = make_float2(mx, se);
            if constexpr (kIdx) sidx[wn * kTM + row] = ai;
          }
        }
    };
    if (a.part_idx)
      rows_pass(std::true_type{});
    else
      rows_pass(std::false_type{});
    __syncthreads();
    if (tid < rows) {
      float m_ = sred[tid].x, s_ = sred[tid].y;
#pragma unroll
      for (int w = 1; w < 4; ++w) lse_merge(m_, s_, sred[w * kTM + tid].x, sred[w * kTM + tid].y);
      a.part[(m0 + tid) * a.n_vt + vt] = make_float2(m_, s_);
      if (a.part_idx) {
        int ai = kNoIdx;
#pragma unroll
        for (int w = 0; w < 4; ++w)
          if (sred[w * kTM + tid].x == m_) ai = min(ai, sidx[w * kTM + tid]);
        a.part_idx[(m0 + tid) * a.n_vt + vt] = ai == kNoIdx ? kNoIdx : int(v0) + ai;
      }
    }
  }
}

// ---------------------------------------------------- MFMA path: prologue
// Per call, before stage 1: (a) per vocabulary tile and column the scale
// ratios of the accumulator's scale slots (residual groups 0 .. d/g-1, then
// s_U if r_c > 0, then s_A if r_r > 0): ratio[vt][k][c] = s'_{k-1} / s'_k
// (0 for k = 0) and fin[vt][c] = s' of the last slot, where s' is the fp16
// scale with zero replaced by kZeroScale; columns past V repeat row V-1;
// (b) the factor codes of V_c and B_w as bf16 (exact), wbf[k][i] for the
// R = r_c + r_r rows; (c) the codes of U_c and A_w side by side per
// vocabulary row, each part zero-padded to a multiple of 16 dimensions, each
// block of 16 stored twice.
struct PrepArgs {
  const uint16_t* rs;
  const uint16_t* rrs;   // row scales of 8-bit group scale codes, or null (fp16 scales)
  const uint16_t* su;
  const uint16_t* sa;
  int64_t V;
  int ngrp, nslot;
  int64_t n_vt;
  float* ratio;
  float* fin;
  const int8_t* cv;
  const int8_t* cb;
  int rc, rr, d;
  uint16_t* wbf;
  const int8_t* cu;
  const int8_t* ca;
  int urow, rc_pad;      // bytes per ucodes row; padded dimensions of the U part
  int8_t* ucodes;
};

__device__ __forceinline__ float nz_scale(uint16_t h) {
  const float s = f16_to_f32(h);
  return s == 0.f ? kZeroScale : s;
}

__global__ __launch_bounds__(kBlock) void k_prep(PrepArgs a) {
  const int64_t nthr = int64_t(gridDim.x) * kBlock;
  const int64_t t0 = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  // (a) one thread per (vocabulary tile, column): walk the slots of the row
  // (lanes write consecutive columns)
  for (int64_t e = t0; e < a.n_vt * kTN; e += nthr) {
    const int64_t vt = e / kTN, c = e % kTN;
    const int64_t v = vt * kTN + c < a.V ? vt * kTN + c : a.V - 1;
    const uint16_t* src = a.rs + v * a.ngrp;
    const uint8_t* src8 = reinterpret_cast<const uint8_t*>(a.rs) + v * a.ngrp;
    const float rsv = a.rrs ? f16_to_f32(a.rrs[v]) : 0.f;
    float* dst = a.ratio + vt * int64_t(a.nslot) * kTN + c;
    float prev = 0.f;
    int k = 0;
    for (; k < a.ngrp; ++k) {
      float s;
      if (a.rrs) {   // rs * q, exact in fp32
        s = rsv * float(src8[k]);
        s = s == 0.f ? kZeroScale : s;
      } else {
        s = nz_scale(src[k]);
      }
      dst[int64_t(k) * kTN] = k ? prev / s : 0.f;
      prev = s;
    }
    if (a.rc) {
      const float s = nz_scale(a.su[v]);
      dst[int64_t(k++) * kTN] = prev / s;
      prev = s;
    }
    if (a.rr) {
      const float s = nz_scale(a.sa[v]);
      dst[int64_t(k++) * kTN] = prev / s;
      prev = s;
    }
    a.fin[vt * kTN + c] = prev;
  }
  // (b) 8 codes per thread
  const int64_t n8 = int64_t(a.rc + a.rr) * a.d / 8;
  for (int64_t e = t0; e < n8; e += nthr) {
    const int64_t k = e * 8 / a.d, i = e * 8 % a.d;
    const int8_t* src = k < a.rc ? a.cv + k * a.d + i : a.cb + (k - a.rc) * a.d + i;
    const uint2 w = *reinterpret_cast<const uint2*>(src);
    uint32_t o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t wj = j < 2 ? w.x : w.y;
      const int sh = 16 * (j & 1);
      const float lo = float(int8_t(wj >> sh)), hi = float(int8_t(wj >> (sh + 8)));
      o[j] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xffff0000u);
    }
    *reinterpret_cast<uint4*>(a.wbf + e * 8) = make_uint4(o[0], o[1], o[2], o[3]);
  }
  // (c) 16 bytes per thread (row-major, so lanes write consecutive chunks)
  const int64_t n16 = a.V * (a.urow / 16);
  for (int64_t e = t0; e < n16; e += nthr) {
    const int64_t v = e / (a.urow / 16);
    const int j0 = int(e % (a.urow / 16)) * 16;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int jj = 0; jj < 16; ++jj) {
      const int j = (j0 / 32) * 16 + jj;   // dimension (both copies of a block)
      int8_t c = 0;
      if (j < a.rc_pad) {
        if (j < a.rc) c = a.cu[v * a.rc + j];
      } else if (j - a.rc_pad < a.rr) {
        c = a.ca[v * a.rr + (j - a.rc_pad)];
      }
      w[jj / 4] |= uint32_t(uint8_t(c)) << (8 * (jj % 4));
    }
    *reinterpret_cast<uint4*>(a.ucodes + v * a.urow + j0) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// ---------------------------------------------------- MFMA path: stage 1
// t[m, k] = sum over factor groups of s[k, grp] * (sum over the group of
// c[k, i] x[m, i]) for the R factor rows (V_c then B_w), and the group biases
// gbias[m / kTM][j][m % kTM] = -136 * (sum of x[m, i] over residual group j)
// (0 for the expansion slots).  t leaves as three bf16 parts hi = bf16(t),
// mid = bf16(t - hi), lo = bf16(t - hi - mid), laid out per block of 16 rank
// dimensions as [hi | mid | lo | 0], the U_c part's blocks first, each part
// zero-padded to whole blocks.
// A workgroup takes 16 tokens and up to 64 factor rows (grid y); its eight
// waves split d by residual groups and each holds 16 x 64 outputs as four
// 16x16 MFMA tiles, loading the next K-chunk's fragments before the current
// chunk's MFMAs; an extra MFMA against a column of ones gives the chunk sums
// of x.  The eight partial results are summed in LDS in a fixed order.
struct Stage1MArgs {
  const uint16_t* x;
  int64_t ldx, M;
  int d, g;
  const uint16_t* wbf;     // [R][d] bf16 factor codes
  const uint16_t* sv;
  int gv, rc;
  const uint16_t* sb;
  int gb, rr;
  uint16_t* tsplit;        // [M][nch][4][16] bf16 (hi, mid, lo, 0)
  int nch, nch_u;
  float* gbias;            // [n_mt][nslot][kTM]
  int nslot;
  int ksplit;              // workgroups along d (grid z); > 1: fp32 partials in tpart
  float* tpart;            // [ksplit][M][R] when ksplit > 1
};

constexpr int kS1MTok = 16, kS1MCols = 64, kS1MBlock = 512, kS1MWaves = kS1MBlock / 64;

__global__ __launch_bounds__(kS1MBlock) void k_stage1m(Stage1MArgs a) {
  __shared__ float red[kS1MWaves][kS1MTok][kS1MCols + 1];
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lr = lane & 15, q = lane >> 4;
  const int R = a.rc + a.rr;
  const int64_t tok0 = int64_t(blockIdx.x) * kS1MTok;
  const int kb = blockIdx.y * kS1MCols;           // first factor row of this workgroup
  const int ngrp = a.d / a.g, cpg = a.g / 32;
  // this workgroup's residual groups (split blockIdx.z of ksplit equal
  // parts), dealt to its waves
  const int ks = blockIdx.z, gps = ngrp / a.ksplit, g0 = ks * gps;
  const int c0 = (g0 + wid * gps / kS1MWaves) * cpg, c1 = (g0 + (wid + 1) * gps / kS1MWaves) * cpg;
  const int64_t mrow = tok0 + lr < a.M ? tok0 + lr : a.M - 1;
  const uint16_t* xrow = a.x + mrow * a.ldx + 8 * q;
  const bool do_bias = blockIdx.y == 0;
  constexpr int NB = kS1MCols / 16;
  const int nblk = R - kb >= kS1MCols ? NB : (R - kb + 15) / 16;

  // this lane's factor row in each 16-column block (clamped; masked on store)
  const uint16_t* wrow[NB];
  const uint16_t* srow[NB];
  int sgrp[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    int k = kb + 16 * nb + lr;
    k = k < R ? k : (R > 0 ? R - 1 : 0);
    wrow[nb] = a.wbf + int64_t(k) * a.d + 8 * q;
    const bool core = k < a.rc;
    sgrp[nb] = core ? a.gv : a.gb;
    srow[nb] = core ? a.sv + int64_t(k) * (a.d / a.gv) : a.sb + int64_t(k - a.rc) * (a.d / a.gb);
  }
  const bf16x8_t ones = {(__bf16)1.f, (__bf16)1.f, (__bf16)1.f, (__bf16)1.f,
                         (__bf16)1.f, (__bf16)1.f, (__bf16)1.f, (__bf16)1.f};
  f32x4_t acc[NB], gs = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  bf16x8_t A, An, B[NB], Bn[NB];
  float s[NB], sn[NB];
  auto load = [&](int c, bf16x8_t& A_, bf16x8_t* B_, float* s_) {
    const int k0 = 32 * c;
    A_ = *reinterpret_cast<const bf16x8_t*>(xrow + k0);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      if (nb < nblk) {
        B_[nb] = *reinterpret_cast<const bf16x8_t*>(wrow[nb] + k0);
        s_[nb] = f16_to_f32(srow[nb][k0 / sgrp[nb]]);
      }
    }
  };
  if (c0 < c1) load(c0, A, B, s);
  for (int c = c0; c < c1; ++c) {
    if (c + 1 < c1) load(c + 1, An, Bn, sn);
    if (do_bias) gs = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, ones, gs, 0, 0, 0);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      if (nb < nblk) {
        const f32x4_t z = {0.f, 0.f, 0.f, 0.f};
        acc[nb] += s[nb] * __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B[nb], z, 0, 0, 0);
      }
    }
    if (do_bias && (c + 1) % cpg == 0) {
      const int j = c / cpg;
      if (lr == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t m = tok0 + 4 * q + i;
          if (m < a.M)
            a.gbias[((m / kTM) * a.nslot + j) * kTM + m % kTM] = -float(archead::kInt4Bias) * gs[i];
        }
      }
      gs = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    A = An;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) B[nb] = Bn[nb], s[nb] = sn[nb];
  }
  if (do_bias && ks == 0) {
    // zero biases of the expansion slots and zero padding of the split t
    const int nz = a.nslot - ngrp;
    for (int e = threadIdx.x; e < kS1MTok * nz; e += kS1MBlock) {
      const int64_t m = tok0 + e / nz;
      if (m < a.M) a.gbias[((m / kTM) * a.nslot + ngrp + e % nz) * kTM + m % kTM] = 0.f;
    }
    const int pu = kExpDims * a.nch_u;   // padded dimensions of the U_c part
    for (int e = threadIdx.x; e < kS1MTok * a.nch * 64; e += kS1MBlock) {
      const int tt = e / (a.nch * 64), j = e % (a.nch * 64), blk = j / 64, w = j % 64;
      const int dim = blk * kExpDims + w % kExpDims;
      const bool pad = w >= 48 || (dim < pu ? dim >= a.rc : dim - pu >= a.rr);
      const int64_t m = tok0 + tt;
      if (m < a.M && pad) a.tsplit[(m * a.nch + blk) * 64 + w] = 0;
    }
  }
  if (R == 0) return;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wid][4 * q + i][16 * nb + lr] = acc[nb][i];
  __syncthreads();
  for (int e = threadIdx.x; e < kS1MTok * kS1MCols; e += kS1MBlock) {
    const int tt = e / kS1MCols, c = e % kS1MCols;
    const int64_t m = tok0 + tt;
    const int k = kb + c;
    if (m < a.M && k < R) {
      float v = red[0][tt][c];
#pragma unroll
      for (int w = 1; w < kS1MWaves; ++w) v += red[w][tt][c];
      if (a.ksplit > 1) {
        a.tpart[(int64_t(ks) * a.M + m) * R + k] = v;
        continue;
      }
      const __bf16 hi = (__bf16)v;
      const float r1 = v - float(hi);
      const __bf16 md = (__bf16)r1;
      const __bf16 lo = (__bf16)(r1 - float(md));
      const int dim = k < a.rc ? k : kExpDims * a.nch_u + (k - a.rc);
      uint16_t* dst = a.tsplit + (m * a.nch + dim / kExpDims) * 64 + dim % kExpDims;
      dst[0] = __builtin_bit_cast(uint16_t, hi);
      dst[16] = __builtin_bit_cast(uint16_t, md);
      dst[32] = __builtin_bit_cast(uint16_t, lo);
    }
  }
}

// t[m][k] as the sum of the ksplit partials in split order, then split
// into three bf16 parts as k_stage1m does when it is not split.
__global__ __launch_bounds__(kBlock) void k_stage1m_fin(Stage1MArgs a) {
  const int R = a.rc + a.rr;
  const int64_t e = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (e >= a.M * R) return;
  const int64_t m = e / R;
  const int k = int(e % R);
  float v = a.tpart[m * R + k];
  for (int ks = 1; ks < a.ksplit; ++ks) v += a.tpart[(int64_t(ks) * a.M + m) * R + k];
  const __bf16 hi = (__bf16)v;
  const float r1 = v - float(hi);
  const __bf16 md = (__bf16)r1;
  const __bf16 lo = (__bf16)(r1 - float(md));
  const int dim = k < a.rc ? k : kExpDims * a.nch_u + (k - a.rc);
  uint16_t* dst = a.tsplit + (m * a.nch + dim / kExpDims) * 64 + dim % kExpDims;
  dst[0] = __builtin_bit_cast(uint16_t, hi);
  dst[16] = __builtin_bit_cast(uint16_t, md);
  dst[32] = __builtin_bit_cast(uint16_t, lo);
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

// Per token: the largest of the partial maxima and the smallest index among
// the partials that hold it (the smallest vocabulary index of the maximum).
__global__ __launch_bounds__(kBlock) void k_argmax_merge(const float2* part, const int* pidx,
                                                         int64_t n_part, int64_t* idx,
                                                         float* max_logit) {
  __shared__ float smx[kBlock];
  __shared__ int sai[kBlock];
  const int64_t m = blockIdx.x;
  float mx = -INFINITY;
  int ai = kNoIdx;
  for (int64_t p = threadIdx.x; p < n_part; p += kBlock) {
    const float v = part[m * n_part + p].x;
    const int i = pidx[m * n_part + p];
    if (v > mx) {
      mx = v;
      ai = i;
    } else if (v == mx) {
      ai = min(ai, i);
    }
  }
  smx[threadIdx.x] = mx;
  sai[threadIdx.x] = ai;
  __syncthreads();
  for (int s = kBlock / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
      const float b = smx[threadIdx.x + s];
      const int bi = sai[threadIdx.x + s];
      if (b > smx[threadIdx.x]) {
        smx[threadIdx.x] = b;
        sai[threadIdx.x] = bi;
      } else if (b == smx[threadIdx.x]) {
        sai[threadIdx.x] = min(sai[threadIdx.x], bi);
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    idx[m] = sai[0] == kNoIdx ? int64_t(-1) : int64_t(sai[0]);
    if (max_logit) max_logit[m] = smx[0];
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
//    into the running fp32 total.
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
#ifndef ARCHEAD_DEC_CPOL
#define ARCHEAD_DEC_CPOL 2
#endif
constexpr int kDecCpol = ARCHEAD_DEC_CPOL;     // cache policy of the code loads

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

// Calls f(integral_constant<J>) for J = I .. N-1 until one returns true.
template <int I, int N, typename F>
__device__ __forceinline__ bool unroll_until(F& f) {
  if constexpr (I < N) {
    if (f(std::integral_constant<int, I>{})) return true;
    return unroll_until<I + 1, N>(f);
  }
  return false;
}

template <int GW, bool CE, int EK, bool SC8>
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
    const int x16 = d / 8;
    for (int e = tid; e < M * x16; e += kDBlock) {
      const int tt = e / x16, u = e - tt * x16;
      *reinterpret_cast<__attribute__((address_space(3))) u32x4_t*>(L + tt * a.xstr + 16 * u) =
          *reinterpret_cast<const u32x4_t*>(a.x + (a.tok0 + tt) * a.ldx + 8 * u);
    }
    __syncthreads();
    auto* sb = reinterpret_cast<__attribute__((address_space(3))) float*>(L + a.off_bias);
    for (int e = tid; e < ngrp * kDTok; e += kDBlock) {
      const int G = e / kDTok, tt = e % kDTok;
      float s = 0.f;
      if (tt < M) {
        const lds_u8* p = L + tt * a.xstr + 2 * G * g;
        for (int i = 0; i < g / 8; ++i) {
          const u32x4_t u = lds_load<u32x4_t>(p + 16 * i);
          s += bf16_lo(u.x) + bf16_hi(u.x) + bf16_lo(u.y) + bf16_hi(u.y) + bf16_lo(u.z) +
               bf16_hi(u.z) + bf16_lo(u.w) + bf16_hi(u.w);
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
  const lds_u8* const xrow = L + xr * a.xstr + 16 * q * GW;
  const lds_u8* const brow = L + a.off_bias + 16 * q;
  const int tpart = M * a.tstr;                        // bf16 elements per part of t in LDS
  const lds_u8* const trow = L + a.off_t + 2 * (xr * a.tstr);
  // this lane's byte offsets within a unit's rows
  const int voff_c = int(uint32_t(lr) * rowbytes) + q * (4 * GW);        // codes: row lr, quarter q
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
        const u32x2_t v = __builtin_amdgcn_raw_buffer_load_b64(lrc, voff_c, so, kDecCpol);
        cbuf[slot][k] = u32x4_t{v.x, v.y, 0u, 0u};
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
      const __amdgpu_buffer_rsrc_t ru = unit_rsrc(a.cu, cu_, uint32_t(a.rc));
      const __amdgpu_buffer_rsrc_t ra = unit_rsrc(a.ca, cu_, uint32_t(a.rr));
#pragma unroll
      for (int kc = 0; kc < EK; ++kc) {
        if (EK == 2 || kc < kcu) eu[kc] = __builtin_amdgcn_raw_buffer_load_b64(ru, voff_u, 8 * kc, 0);
        if (EK == 2 || kc < kca) ea[kc] = __builtin_amdgcn_raw_buffer_load_b64(ra, voff_a, 8 * kc, 0);
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
#pragma unroll
      for (int kc = 0; kc < GW; ++kc) {
#pragma unroll
        for (int k = 0; k < SG; ++k) {
          const bf16x8_t A = lds_load<bf16x8_t>(xrow + 2 * (cS * SG + k) * g + 16 * kc);
          acc[k] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              A, unpack8(cbuf[j][k][kc], kMask, kMagic), acc[k], 0, 0, 0);
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

// ------------------------------------------------- several-token kernel
// k_mid: the tokens of a call in tiles of TM = 16 NF (NF MFMA row blocks);
// the head is streamed once per tile.  A consumer workgroup owns a
// contiguous, balanced range of 16-row units; its eight waves take the units
// in turn, NU at a time (a pass), and hold the accumulators of all of them.
// x of a tile does not fit LDS whole, so the workgroup walks d in windows of
// kMidKW elements in lock-step: every thread fetches its share of a window
// into registers two windows ahead, and at the end of the window before it
// writes that share, with the per-group offset biases (-136 times the sum
// of x over the group, summed across the lanes holding the group with DPP),
// to the other LDS buffer before the window's closing barrier.  Codes arrive
// as in k_dec (lane (j, q): row j of the unit, GW dwords from q GW of each
// group) for all NU units at once, a 128-byte line of each row per request
// round, one line ahead; a unit's group partial starts from the bias (MFMA
// C input) and is scaled into the unit's total.  After the last window of a pass the window buffers hold t (three
// bf16 parts) for the rank-r expansion, then the units' logits go out.
// Stage 1 (t) runs in the same launch as in k_dec.
constexpr int kMidBlock = 512, kMidWaves = kMidBlock / 64;
constexpr int kMidKW = 256;   // elements of d per x window
constexpr int kMidXstr = 2 * kMidKW + 16;   // LDS bytes per token row of a window
static_assert(kMidKW == archead::kMidWindow && kMidWaves == archead::kMidWaveCount,
              "host and kernel agree on the window and the workgroup");

struct MidArgs {
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
  int64_t tok0;          // first token of this tile
  int M;                 // tokens of this tile (1 .. 16 NF)
  int64_t V;
  int d, rc, rr, ngrp, kcu, kca;
  int64_t n_units;       // ceil(V / 16)
  int n_cblocks;         // consumer workgroups
  int n_prod_blocks;     // leading workgroups that compute t
  int tstr;              // LDS: bf16 elements per token row of each part of t
  int off_bias, off_red, off_y, off_idx, off_sc;   // LDS byte offsets
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

__device__ __forceinline__ float row8_sum(float v) {
  v += dpp_swap<0xB1>(v);
  v += dpp_swap<0x4E>(v);
  return v + dpp_swap<0x141>(v);
}

// LDS writes done, then the workgroup meets (loads in flight stay in flight)
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int GW, int NF, int NU, bool CE, bool SC8>
__global__ __launch_bounds__(kMidBlock) __attribute__((amdgpu_waves_per_eu(2)))
void k_mid(MidArgs a) {
  static_assert(GW == 2 || GW == 4, "groups of 64 or 128 codes");
  constexpr int TM = 16 * NF;
  constexpr int G = 32 * GW;                  // group size
  constexpr int SPW = kMidKW / G;             // groups per window
  // Code loads go out a 128-byte line of each row at a time (LG groups:
  // both halves of a line are requested together, not a step apart), one
  // line ahead, so the ring holds two lines of groups
  constexpr int LG = 256 / G;
  constexpr int NB = 2 * LG;
  static_assert((2 * SPW) % NB == 0, "ring slots are compile-time per step");
  extern __shared__ __align__(16) uint8_t mid_lds[];
  lds_u8* const L = (lds_u8*)mid_lds;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, q = lane >> 4;
  const int M = a.M, d = a.d, ngrp = a.ngrp;
  const int R = a.rc + a.rr;

  // ---- stage-1 producers: one rank row per wave, the tile's tokens in
  // blocks of 16, x read from memory
  if (int(blockIdx.x) < a.n_prod_blocks) {
    const int k = int(blockIdx.x) * kMidWaves + wid;
    if (k < R) {
#pragma unroll 1
      for (int f = 0; f < NF; ++f) {
        const int m0 = 16 * f;
        if (m0 >= M) break;
        const uint16_t* xb = a.x + (a.tok0 + m0) * a.ldx;
        const int64_t ldx = a.ldx;
        s1_produce<16>(a.s1, k, M - m0 < 16 ? M - m0 : 16, a.tok0 + m0,
                       [&](int tt, int i) {
                         return *reinterpret_cast<const u32x4_t*>(xb + tt * ldx + i);
                       },
                       lane);
      }
    }
    return;
  }

  // ---- consumers
  const int cb = int(blockIdx.x) - a.n_prod_blocks;
  const int64_t u_lo = a.n_units * cb / a.n_cblocks;
  const int nub = int(a.n_units * (cb + 1) / a.n_cblocks - u_lo);   // units of the workgroup
  const int n_pass = (nub + kMidWaves * NU - 1) / (kMidWaves * NU);
  const int nwin = d / kMidKW;
  const uint32_t rowbytes = uint32_t(d) / 2;
  const uint32_t kMask = opaque_vgpr(0x000F000Fu);
  const uint32_t kMagic = opaque_vgpr(0x43004300u);
  const int kcu = a.kcu, kca = a.kca;
  // this lane's byte offsets within a unit's rows
  const int voff_c = int(uint32_t(lr) * rowbytes) + q * (4 * GW);   // codes: row lr, part q
  const int voff_u = lr * a.rc + q * (8 * kcu);
  const int voff_a = lr * a.rr + q * (8 * kca);
  auto* const sbias = reinterpret_cast<__attribute__((address_space(3))) float*>(L + a.off_bias);
  float2* const sred = reinterpret_cast<float2*>(mid_lds + a.off_red);
  int64_t* const sy = reinterpret_cast<int64_t*>(mid_lds + a.off_y);
  int* const sidx = reinterpret_cast<int*>(mid_lds + a.off_idx);   // [waves][TM] argmax
  // residual scales of this wave's units: [unit][row][group] fp16 (8-bit
  // codes widened to fp16, exact), rows padded by 4 bytes so the 16 rows
  // read at one step fall on distinct banks
  const int sstr = 2 * ngrp + 4;
  lds_u8* const ssc = L + a.off_sc + wid * (NU * 16 * sstr);
  if constexpr (CE) {
    for (int e = tid; e < kMidWaves * TM; e += kMidBlock) {
      sred[e] = make_float2(-INFINITY, 0.f);
      sidx[e] = kNoIdx;
    }
    for (int e = tid; e < TM; e += kMidBlock)
      sy[e] = e >= M || !a.tgt
                  ? int64_t(-1)
                  : (a.tgt64 ? reinterpret_cast<const int64_t*>(a.tgt)[a.tok0 + e]
                             : int64_t(reinterpret_cast<const int32_t*>(a.tgt)[a.tok0 + e]));
  }

  // buffer resource over the rows of unit u of an array with `stride` bytes
  // per vocabulary row (rows past V read as zero; a unit past the head has
  // no rows)
  auto unit_rsrc = [&](const void* base, int64_t u, uint32_t stride) {
    const int64_t v0 = u * 16;
    const int64_t left = a.V - v0;
    const uint32_t rows = uint32_t(left <= 0 ? 0 : (left < 16 ? left : 16));
    return __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(static_cast<const char*>(base)) + (rows ? v0 * stride : 0), 0,
        int(rows * stride), kBufferWord3);
  };

  // x window w of the tile: thread tid holds the 16-byte pieces tid + 512 i
  // (token row tid / 32 + 16 i, elements 8 (tid % 32) ..), rows past the
  // tile repeat its last row.  Two register sets: a window is fetched two
  // windows before it is computed.
  u32x4_t xr[2][NF];
  auto load_win = [&](auto SET, int w) {
    constexpr int set = decltype(SET)::value;
    w = w < nwin ? w : nwin - 1;
#pragma unroll
    for (int i = 0; i < NF; ++i) {
      const int row = (tid >> 5) + 16 * i;
      const int rw = row < M ? row : M - 1;
      xr[set][i] = *reinterpret_cast<const u32x4_t*>(a.x + (a.tok0 + rw) * a.ldx + w * kMidKW +
                                                      8 * (tid & 31));
    }
  };
  auto store_win = [&](auto SET, int w) {
    constexpr int set = decltype(SET)::value;
    lds_u8* const xb = L + (w & 1) * (TM * kMidXstr);
    auto* const bb = sbias + (w & 1) * (SPW * TM);
    const int c16 = tid & 31;
#pragma unroll
    for (int i = 0; i < NF; ++i) {
      const int row = (tid >> 5) + 16 * i;
      const u32x4_t v = xr[set][i];
      *reinterpret_cast<__attribute__((address_space(3))) u32x4_t*>(xb + row * kMidXstr + 16 * c16) = v;
      float sm = ((bf16_lo(v.x) + bf16_hi(v.x)) + (bf16_lo(v.y) + bf16_hi(v.y))) +
                 ((bf16_lo(v.z) + bf16_hi(v.z)) + (bf16_lo(v.w) + bf16_hi(v.w)));
      sm = GW == 4 ? row16_sum(sm) : row8_sum(sm);
      if ((c16 & (4 * GW - 1)) == 0) bb[(c16 / (4 * GW)) * TM + row] = -float(archead::kInt4Bias) * sm;
    }
  };

  // t of the tile's tokens (from the producers) into LDS as three bf16
  // parts over the window buffers, zero in the padding dimensions.  The
  // stamped words are read eight per thread at a time; a value whose stamp
  // is not there yet goes through the bounded wait (and its fallback).
  const int tw = 32 * (kcu + kca);
  const int tpart = TM * a.tstr;
  auto fetch_t = [&]() {
    auto* st = reinterpret_cast<__attribute__((address_space(3))) uint16_t*>(L);
    const int n = TM * tw;
    const uint16_t* xt = a.x + a.tok0 * a.ldx;
    const int64_t ldx = a.ldx;
    for (int e0 = tid; e0 < n; e0 += 8 * kMidBlock) {
      unsigned long long wv[8];
      int kk[8];
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        const int e = e0 + b * kMidBlock;
        const int tt = e / tw, c = e - tt * tw;
        int k = -1;
        if (c < 32 * kcu) {
          if (c < a.rc) k = c;
        } else if (c - 32 * kcu < a.rr) {
          k = a.rc + (c - 32 * kcu);
        }
        kk[b] = (e < n && tt < M) ? k : -1;
        const int ta = tt < M ? tt : M - 1;
        wv[b] = load_stamped(a.s1.tst + (a.tok0 + ta) * R + (k >= 0 ? k : 0));
      }
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        const int e = e0 + b * kMidBlock;
        if (e >= n) break;
        const int tt = e / tw, c = e - tt * tw;
        float v = 0.f;
        if (kk[b] >= 0) {
          v = uint32_t(wv[b] >> 32) == a.s1.epoch
                  ? __uint_as_float(uint32_t(wv[b]))
                  : s1_value(a.s1, a.tok0, tt, kk[b], [&](int t2, int i) {
                      return *reinterpret_cast<const uint32_t*>(xt + t2 * ldx + i);
                    });
        }
        const __bf16 hi = (__bf16)v;
        const float r1 = v - float(hi);
        const __bf16 md = (__bf16)r1;
        const __bf16 lo = (__bf16)(r1 - float(md));
        const int o = tt * a.tstr + c;
        st[o] = __builtin_bit_cast(uint16_t, hi);
        st[tpart + o] = __builtin_bit_cast(uint16_t, md);
        st[2 * tpart + o] = __builtin_bit_cast(uint16_t, lo);
      }
    }
  };

  u32x4_t cbuf[NB][NU];
  __amdgpu_buffer_rsrc_t rcu[NU];
  auto load_step = [&](auto SLOT, int s) {
    constexpr int slot = decltype(SLOT)::value;
#pragma unroll
    for (int j = 0; j < NU; ++j) {
      if constexpr (GW == 4) {
        cbuf[slot][j] = __builtin_amdgcn_raw_buffer_load_b128(rcu[j], voff_c, s * (G / 2), kDecCpol);
      } else {
        const u32x2_t v = __builtin_amdgcn_raw_buffer_load_b64(rcu[j], voff_c, s * (G / 2), kDecCpol);
        cbuf[slot][j] = u32x4_t{v.x, v.y, 0u, 0u};
      }
    }
  };
  // absent factors: stride-0 resources over valid buffers (read as zero)
  const void* const cu_b = a.rc ? static_cast<const void*>(a.cu) : static_cast<const void*>(a.rs);
  const void* const ca_b = a.rr ? static_cast<const void*>(a.ca) : static_cast<const void*>(a.rs);
  const void* const su_b = a.rc ? static_cast<const void*>(a.su) : static_cast<const void*>(a.rs);
  const void* const sa_b = a.rr ? static_cast<const void*>(a.sa) : static_cast<const void*>(a.rs);

#pragma unroll 1
  for (int p = 0; p < n_pass; ++p) {
    int64_t uj[NU];
#pragma unroll
    for (int j = 0; j < NU; ++j) {
      const int ui = p * (kMidWaves * NU) + wid + kMidWaves * j;
      uj[j] = ui < nub ? u_lo + ui : a.n_units;   // past the head: no rows
      rcu[j] = unit_rsrc(a.codes, uj[j], rowbytes);
    }
    // the units' scales (pieces of 4 groups: 8 bytes of fp16 or 4 bytes of
    // 8-bit codes, issued first so that waiting for them leaves the code
    // loads in flight), the pass's first code loads, the first two windows
    {
      using Piece = typename std::conditional<SC8, uint32_t, u32x2_t>::type;
      Piece sp[NU][4];
#pragma unroll
      for (int j = 0; j < NU; ++j) {
        const __amdgpu_buffer_rsrc_t r_ = unit_rsrc(a.rs, uj[j], uint32_t((SC8 ? 1 : 2) * ngrp));
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if constexpr (SC8)
            sp[j][i] = __builtin_amdgcn_raw_buffer_load_b32(r_, 4 * (lane + 64 * i), 0, 0);
          else
            sp[j][i] = __builtin_amdgcn_raw_buffer_load_b64(r_, 8 * (lane + 64 * i), 0, 0);
        }
      }
      load_win(std::integral_constant<int, 0>{}, 0);
      load_win(std::integral_constant<int, 1>{}, 1);
      load_step(std::integral_constant<int, 0>{}, 0);
      load_step(std::integral_constant<int, 1>{}, 1);
      if constexpr (LG == 4) {
        load_step(std::integral_constant<int, 2>{}, 2);
        load_step(std::integral_constant<int, 3>{}, 3);
      }
      const int pr = ngrp / 4;   // pieces per row
#pragma unroll
      for (int j = 0; j < NU; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int pc = lane + 64 * i;
          if (pc < 16 * pr) {
            const int row = pc / pr, c = pc - row * pr;
            auto* dst = reinterpret_cast<__attribute__((address_space(3))) uint32_t*>(
                ssc + (j * 16 + row) * sstr + 8 * c);
            u32x2_t pv;
            if constexpr (SC8)
              pv = u8x4_to_f16x4(sp[j][i]);
            else
              pv = sp[j][i];
            dst[0] = pv.x;
            dst[1] = pv.y;
          }
        }
    }
    store_win(std::integral_constant<int, 0>{}, 0);
    lds_barrier();

    f32x4_t tot[NU][NF];
#pragma unroll
    for (int j = 0; j < NU; ++j)
#pragma unroll
      for (int f = 0; f < NF; ++f) tot[j][f] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // iterations of two windows (2 SPW groups): window parity and ring slot
    // of every step are compile-time constants
    constexpr int IT = 2 * SPW;
#pragma unroll 1
    for (int it = 0; it < ngrp / IT; ++it) {
      auto body = [&](auto J) {
        constexpr int j = decltype(J)::value;
        constexpr int par = j / SPW;             // window parity (set of its fetch)
        const int s = IT * it + j;               // group of this step
        const int w = 2 * it + par;              // its window
        if constexpr (j % SPW == 0) load_win(std::integral_constant<int, par>{}, w + 2);
        if constexpr (j % LG == 0) {
          // the next line of every row: groups s + LG .. s + 2 LG - 1
          auto next = [&](auto E) {
            constexpr int e = decltype(E)::value;
            const int sn = s + LG + e;
            load_step(std::integral_constant<int, (j + LG + e) % NB>{}, sn < ngrp ? sn : ngrp - 1);
          };
          next(std::integral_constant<int, 0>{});
          next(std::integral_constant<int, 1>{});
          if constexpr (LG == 4) {
            next(std::integral_constant<int, 2>{});
            next(std::integral_constant<int, 3>{});
          }
        }
        asm volatile("" ::: "memory");
        const lds_u8* const xb = L + par * (TM * kMidXstr) + (j % SPW) * (2 * G);
        const auto* bb = sbias + par * (SPW * TM) + (j % SPW) * TM;
        f32x4_t acc[NU][NF];
#pragma unroll
        for (int kc = 0; kc < GW; ++kc) {
          bf16x8_t A[NF];
#pragma unroll
          for (int f = 0; f < NF; ++f)
            A[f] = lds_load<bf16x8_t>(xb + (16 * f + lr) * kMidXstr + 16 * (q * GW + kc));
#pragma unroll
          for (int u = 0; u < NU; ++u) {
            const bf16x8_t B = unpack8(cbuf[j % NB][u][kc], kMask, kMagic);
#pragma unroll
            for (int f = 0; f < NF; ++f) {
              const f32x4_t c0 =
                  kc == 0 ? *reinterpret_cast<const __attribute__((address_space(3))) f32x4_t*>(
                                bb + 16 * f + 4 * q)
                          : acc[u][f];
              acc[u][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[f], B, c0, 0, 0, 0);
            }
          }
          // one K-chunk's fragments live at a time (the scheduler would
          // otherwise hoist every chunk's LDS reads and unpacks, past the
          // register budget)
          __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int u = 0; u < NU; ++u) {
          const float sc = f16_to_f32(lds_load<uint16_t>(ssc + (u * 16 + lr) * sstr + 2 * s));
#pragma unroll
          for (int f = 0; f < NF; ++f) tot[u][f] += sc * acc[u][f];
        }
        if constexpr (j % SPW == SPW - 1) {
          // window w + 1 (fetched during window w - 1, or before the loop)
          store_win(std::integral_constant<int, 1 - par>{}, w + 1);
          lds_barrier();
        }
      };
      body(std::integral_constant<int, 0>{});
      body(std::integral_constant<int, 1>{});
      body(std::integral_constant<int, 2>{});
      body(std::integral_constant<int, 3>{});
      if constexpr (IT == 8) {
        body(std::integral_constant<int, 4>{});
        body(std::integral_constant<int, 5>{});
        body(std::integral_constant<int, 6>{});
        body(std::integral_constant<int, 7>{});
      }
    }

    // ---- rank-r expansion and the units' logits.  Its operands are
    // requested together, then t goes to LDS while they are in flight.
    u32x2_t eu[NU][4], ea[NU][4];
    uint16_t esu[NU], esa[NU];
    uint16_t ers[NU];   // row scales of 8-bit residual scale codes
#pragma unroll
    for (int j = 0; j < NU; ++j) {
      const __amdgpu_buffer_rsrc_t ru = unit_rsrc(cu_b, uj[j], uint32_t(a.rc));
      const __amdgpu_buffer_rsrc_t ra = unit_rsrc(ca_b, uj[j], uint32_t(a.rr));
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) {
        eu[j][kc] = __builtin_amdgcn_raw_buffer_load_b64(ru, voff_u, 8 * kc, 0);
        ea[j][kc] = __builtin_amdgcn_raw_buffer_load_b64(ra, voff_a, 8 * kc, 0);
      }
      esu[j] = __builtin_amdgcn_raw_buffer_load_b16(unit_rsrc(su_b, uj[j], a.rc ? 2u : 0u), 2 * lr, 0, 0);
      esa[j] = __builtin_amdgcn_raw_buffer_load_b16(unit_rsrc(sa_b, uj[j], a.rr ? 2u : 0u), 2 * lr, 0, 0);
      if constexpr (SC8)
        ers[j] = __builtin_amdgcn_raw_buffer_load_b16(unit_rsrc(a.rrs, uj[j], 2u), 2 * lr, 0, 0);
    }
    lds_barrier();          // every wave is done with the windows
    if (R > 0) {
      fetch_t();
      lds_barrier();
    }
#pragma unroll
    for (int j = 0; j < NU; ++j) {
      if (uj[j] >= a.n_units) continue;
      if constexpr (SC8) {   // the residual was summed in units of the row scale
        const float fr = f16_to_f32(ers[j]);
#pragma unroll
        for (int f = 0; f < NF; ++f) tot[j][f] *= fr;
      }
      if (kcu + kca > 0) {
        f32x4_t au[NF], aa[NF];
#pragma unroll
        for (int f = 0; f < NF; ++f) {
          au[f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
          aa[f] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) {
          if (kc < kcu) {
            const bf16x8_t B = int8x8_to_bf16(eu[j][kc].x, eu[j][kc].y);
#pragma unroll
            for (int f = 0; f < NF; ++f) {
              const lds_u8* tp = L + 2 * ((16 * f + lr) * a.tstr + q * 8 * kcu + 8 * kc);
#pragma unroll
              for (int pp = 0; pp < 3; ++pp)
                au[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    lds_load<bf16x8_t>(tp + 2 * pp * tpart), B, au[f], 0, 0, 0);
            }
          }
          if (kc < kca) {
            const bf16x8_t B = int8x8_to_bf16(ea[j][kc].x, ea[j][kc].y);
#pragma unroll
            for (int f = 0; f < NF; ++f) {
              const lds_u8* tp = L + 2 * ((16 * f + lr) * a.tstr + 32 * kcu + q * 8 * kca + 8 * kc);
#pragma unroll
              for (int pp = 0; pp < 3; ++pp)
                aa[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    lds_load<bf16x8_t>(tp + 2 * pp * tpart), B, aa[f], 0, 0, 0);
            }
          }
          __builtin_amdgcn_sched_barrier(0);
        }
        const float fu = f16_to_f32(esu[j]), fa = f16_to_f32(esa[j]);
#pragma unroll
        for (int f = 0; f < NF; ++f) tot[j][f] += fu * au[f] + fa * aa[f];
      }
      const int64_t v = uj[j] * 16 + lr;
      const bool vok = v < a.V;
#pragma unroll
      for (int f = 0; f < NF; ++f) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int tt = 16 * f + 4 * q + r;
          const float l = tot[j][f][r];
          if constexpr (!CE) {
            if (tt < M && vok) {
              const int64_t o = (a.tok0 + tt) * a.ldo + v;
              if (a.out_bf16)
                reinterpret_cast<uint16_t*>(a.out)[o] = f32_to_bf16_rne(l);
              else
                reinterpret_cast<float*>(a.out)[o] = l;
            }
          } else {
            const float m = row16_max(vok ? l : -INFINITY);
            const float e = row16_sum(vok ? fast_exp(l - m) : 0.f);
            const int ai = row16_min_i(vok && l == m ? int(v) : kNoIdx);
            if (vok && tt < M && v == sy[tt]) a.tgt_logit[a.tok0 + tt] = l;
            if (lr == 0) {
              float2 cur = sred[wid * TM + tt];
              const int ci = sidx[wid * TM + tt];
              sidx[wid * TM + tt] = m > cur.x ? ai : (m == cur.x ? min(ci, ai) : ci);
              lse_merge(cur.x, cur.y, m, e);
              sred[wid * TM + tt] = cur;
            }
          }
        }
      }
    }
    if (p + 1 < n_pass) lds_barrier();   // t is overwritten by the next pass's windows
  }

  if constexpr (CE) {
    lds_barrier();
    if (tid < M) {
      float m = sred[tid].x, s = sred[tid].y;
      for (int w = 1; w < kMidWaves; ++w) lse_merge(m, s, sred[w * TM + tid].x, sred[w * TM + tid].y);
      a.part[(a.tok0 + tid) * a.n_part + cb] = make_float2(m, s);
      if (a.part_idx) {
        int ai = kNoIdx;
        for (int w = 0; w < kMidWaves; ++w)
          if (sred[w * TM + tid].x == m) ai = min(ai, sidx[w * TM + tid]);
        a.part_idx[(a.tok0 + tid) * a.n_part + cb] = ai;
      }
    }
  }
}

// ------------------------------------------------------------ dispatch
using GemvFn = void (*)(GemvArgs);

template <int TOK, bool CE, bool SC8>
GemvFn gemv_by_lpr(int lpr) {
  switch (lpr) {
    case 1: return k_gemv<TOK, 1, CE, SC8>;
    case 2: return k_gemv<TOK, 2, CE, SC8>;
    case 4: return k_gemv<TOK, 4, CE, SC8>;
    case 8: return k_gemv<TOK, 8, CE, SC8>;
    case 16: return k_gemv<TOK, 16, CE, SC8>;
    case 32: return k_gemv<TOK, 32, CE, SC8>;
    default: return k_gemv<TOK, 64, CE, SC8>;
  }
}

template <bool CE, bool SC8>
GemvFn gemv_fn_sc(int tok, int lpr) {
  switch (tok) {
    case 1: return gemv_by_lpr<1, CE, SC8>(lpr);
    case 2: return gemv_by_lpr<2, CE, SC8>(lpr);
    case 3: return gemv_by_lpr<3, CE, SC8>(lpr);
    default: return gemv_by_lpr<4, CE, SC8>(lpr);
  }
}

// the variant for the head's residual scale format (8-bit codes or fp16)
template <bool CE>
GemvFn gemv_fn(int tok, int lpr, bool sc8) {
  return sc8 ? gemv_fn_sc<CE, true>(tok, lpr) : gemv_fn_sc<CE, false>(tok, lpr);
}

size_t gemv_lds_bytes(const archead_desc& d, int tok) {
  // x, the chunk biases, and one copy of t per wave
  return size_t(tok) * (size_t(d.d) * 2 + size_t(d.d / 32) * 4 +
                        size_t(kWaves) * size_t(d.r_c + d.r_r) * 4);
}

int64_t gemv_rows_per_step(const archead_desc& d) {
  const int lpr = archead::lanes_per_row(d);
  return int64_t(lpr < kRowsPerStep ? lpr : kRowsPerStep) * (64 / lpr);
}

archead_status hip_fail(hipError_t e, const char* what) {
  return archead::fail(ARCHEAD_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

namespace archead {

int64_t gemv_grid(const archead_handle* h, int tok, bool ce) {
  const bool sc8 = h->desc.scale_dtype == ARCHEAD_U8;
  const int slot = (sc8 ? 16 : 0) + (ce ? 8 : 0) + tok;
  archead_handle* mh = const_cast<archead_handle*>(h);
  int cached = mh->grid_cache[slot].load(std::memory_order_relaxed);
  const int64_t steps = (h->desc.V + gemv_rows_per_step(h->desc) - 1) / gemv_rows_per_step(h->desc);
  const int64_t max_blocks = (steps + kWaves - 1) / kWaves;
  if (cached <= 0) {
    const int lpr = lanes_per_row(h->desc);
    GemvFn fn = ce ? gemv_fn<true>(tok, lpr, sc8) : gemv_fn<false>(tok, lpr, sc8);
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
    // every resident wave (measured faster than fewer waves with an even
    // split of the steps)
    cached = nb * h->n_cu;
    if (const char* e = getenv("ARCHEAD_GEMV_GRID")) cached = atoi(e) > 0 ? atoi(e) : cached;
    mh->grid_cache[slot].store(cached, std::memory_order_relaxed);
  }
  return cached < max_blocks ? cached : max_blocks;
}

// MFMA decode kernel grid: stage-1 producer workgroups (one rank row per
// wave) first, then one consumer workgroup per remaining CU at most, with
// the consumer wave count chosen so the 16-row units divide evenly into
// rounds (every wave gets the same number of units, but for the last round).
DecGrid dec_grid(const archead_handle* h) {
  DecGrid gr;
  const archead_desc& d = h->desc;
  const int64_t R = d.r_c + d.r_r;
  gr.prod_blocks = int((R + kDecWaves - 1) / kDecWaves);
  gr.n_units = (d.V + 15) / 16;
  int64_t cap = int64_t(h->n_cu) - gr.prod_blocks;
  if (cap < 1) cap = 1;
  if (const char* e = getenv("ARCHEAD_DEC_BLOCKS")) cap = atoi(e) > 0 ? atoi(e) : cap;
  const int64_t wmax = cap * kDecWaves;
  const int64_t rounds = (gr.n_units + wmax - 1) / wmax;
  gr.n_waves = (gr.n_units + rounds - 1) / rounds;
  gr.consumer_blocks = (gr.n_waves + kDecWaves - 1) / kDecWaves;
  return gr;
}

// Several-token kernel grid: stage-1 producer workgroups first, then one
// consumer workgroup per remaining CU, each with a balanced contiguous range
// of 16-row units (at least one unit each).
MidGrid mid_grid(const archead_handle* h) {
  MidGrid gr;
  const archead_desc& d = h->desc;
  const int64_t R = d.r_c + d.r_r;
  gr.prod_blocks = int((R + kMidWaveCount - 1) / kMidWaveCount);
  gr.n_units = (d.V + 15) / 16;
  int64_t cap = int64_t(h->n_cu) - gr.prod_blocks;
  if (cap < 1) cap = 1;
  if (const char* e = getenv("ARCHEAD_MID_BLOCKS")) cap = atoi(e) > 0 ? atoi(e) : cap;
  gr.cblocks = cap < gr.n_units ? cap : gr.n_units;
  return gr;
}

static size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int exp_chunks(int64_t r) { return int((r + kExpDims - 1) / kExpDims); }   // stages per part

// The many-token kernel stages 64 codes of one scale group at a time.
static bool mfma_ok(const archead_handle* h) { return h->desc.g % 64 == 0; }

// Workgroups along d of the tiled path's stage 1: doubled (while every wave
// keeps at least one residual group and the groups split evenly) until the
// grid has 256 workgroups, so a call with few token blocks still spreads
// the factor-code reads over the chip.
static int s1_ksplit(const archead_handle* h, int64_t M) {
  const archead_desc& d = h->desc;
  const int64_t R = d.r_c + d.r_r;
  if (R == 0 || M <= 0) return 1;
  const int64_t ngrp = d.d / d.g;
  const int64_t blocks = ((M + kS1MTok - 1) / kS1MTok) * ((R + kS1MCols - 1) / kS1MCols);
  int ks = 1;
  while (blocks * ks < 256 && ngrp % (2 * ks) == 0 && ngrp / (2 * ks) >= kS1MWaves) ks *= 2;
  return ks;
}

PrepLayout prep_layout(const archead_handle* h) {
  PrepLayout p;
  if (!h) return p;
  const archead_desc& d = h->desc;
  const size_t ngrp = size_t(d.d / d.g);
  const size_t nslot = ngrp + (d.r_c ? 1 : 0) + (d.r_r ? 1 : 0);
  const size_t nch = size_t(exp_chunks(d.r_c) + exp_chunks(d.r_r));
  const size_t n_vt = size_t((d.V + kTN - 1) / kTN);
  size_t off = 0;
  p.rat_off = off;
  off = align256(off + sizeof(float) * n_vt * nslot * kTN);
  p.fin_off = off;
  off = align256(off + sizeof(float) * n_vt * kTN);
  p.wbf_off = off;
  off = align256(off + sizeof(uint16_t) * size_t(d.r_c + d.r_r) * size_t(d.d));
  p.uc_off = off;
  off = align256(off + size_t(d.V) * nch * 32);                    // [c|c] x 16
  p.total = off;
  return p;
}

WsLayout ws_layout(const archead_handle* h, int64_t M, archead_op op) {
  WsLayout w;
  if (!h || M <= 0) return w;
  const archead_desc& d = h->desc;
  size_t off = 0;
  const Path path = choose_path(h, M);
  const bool dec = path == Path::kDec, mid = path == Path::kMid, gemv = path == Path::kGemv;
  if (dec || mid) {
    w.tst_off = off;
    off = align256(off + sizeof(uint64_t) * size_t(M) * size_t(d.r_c + d.r_r));
  } else if (gemv) {
    w.tst_off = off;
    off = align256(off + sizeof(uint64_t) * size_t(M) * size_t(d.r_c + d.r_r));
  } else {
    const size_t ngrp = size_t(d.d / d.g);
    const size_t nslot = ngrp + (d.r_c ? 1 : 0) + (d.r_r ? 1 : 0);
    const size_t nch = size_t(exp_chunks(d.r_c) + exp_chunks(d.r_r));
    const size_t n_mt = size_t((M + kTM - 1) / kTM);
    w.ts_off = off;
    off = align256(off + sizeof(uint16_t) * size_t(M) * nch * 64);   // [hi|mid|lo|0] x 16
    w.gb_off = off;
    off = align256(off + sizeof(float) * n_mt * nslot * kTM);
    const PrepLayout pl = prep_layout(h);
    w.rat_off = off + pl.rat_off;
    w.fin_off = off + pl.fin_off;
    w.wbf_off = off + pl.wbf_off;
    w.uc_off = off + pl.uc_off;
    off += pl.total;
    const int ks = s1_ksplit(h, M);
    if (ks > 1) {
      w.s1p_off = off;
      off = align256(off + sizeof(float) * size_t(ks) * size_t(M) * size_t(d.r_c + d.r_r));
    }
  }
  if (op == ARCHEAD_OP_LOGITS_CE || op == ARCHEAD_OP_ARGMAX) {
    // GEMV: all CE passes share one grid (the smallest of the variants
    // used) so every token row of the partials has the same number of
    // slots.  MFMA: one slot per vocabulary tile.
    int64_t np = 0;
    if (dec) {
      np = dec_grid(h).consumer_blocks;
    } else if (mid) {
      np = mid_grid(h).cblocks;
    } else if (gemv) {
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
    if (op == ARCHEAD_OP_ARGMAX) {
      w.pidx_off = off;
      off = align256(off + sizeof(int32_t) * size_t(M) * size_t(np));
    }
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

// Start of the block of head-derived tables a call of the many-token
// kernel reads: the prepared buffer when the head has one, else the call's
// workspace.
char* prep_base(const archead_handle* h, const WsLayout& w, char* ws) {
  char* p = h->prep.load(std::memory_order_acquire);
  return p ? p : ws + w.rat_off;
}

// The head-derived tables (tile-major residual scale ratios, final scales,
// bf16 factor codes of V_c / B_w, paired U_c / A_w codes) into the block at
// base, laid out as prep_layout says.
archead_status launch_prep(const archead_handle* h, char* base, hipStream_t s) {
  const archead_desc& d = h->desc;
  const PrepLayout pl = prep_layout(h);
  const int R = int(d.r_c + d.r_r);
  const int nch_u = exp_chunks(d.r_c), nch = nch_u + exp_chunks(d.r_r);
  PrepArgs p;
  p.rs = static_cast<const uint16_t*>(h->ptrs.res_scales);
  p.rrs = d.scale_dtype == ARCHEAD_U8 ? static_cast<const uint16_t*>(h->ptrs.res_row_scales)
                                      : nullptr;
  p.su = static_cast<const uint16_t*>(h->ptrs.core_u_scale);
  p.sa = static_cast<const uint16_t*>(h->ptrs.corr_a_scale);
  p.V = d.V;
  p.ngrp = int(d.d / d.g);
  p.nslot = p.ngrp + (d.r_c ? 1 : 0) + (d.r_r ? 1 : 0);
  p.n_vt = (d.V + kTN - 1) / kTN;
  p.ratio = reinterpret_cast<float*>(base + pl.rat_off);
  p.fin = reinterpret_cast<float*>(base + pl.fin_off);
  p.cv = static_cast<const int8_t*>(h->ptrs.core_v);
  p.cb = static_cast<const int8_t*>(h->ptrs.corr_b);
  p.rc = int(d.r_c); p.rr = int(d.r_r); p.d = int(d.d);
  p.wbf = reinterpret_cast<uint16_t*>(base + pl.wbf_off);
  p.cu = static_cast<const int8_t*>(h->ptrs.core_u);
  p.ca = static_cast<const int8_t*>(h->ptrs.corr_a);
  p.urow = nch * 32;
  p.rc_pad = nch_u * kExpDims;
  p.ucodes = reinterpret_cast<int8_t*>(base + pl.uc_off);
  const int64_t work = std::max({p.n_vt * kTN, int64_t(R) * d.d / 8, d.V * (p.urow / 16)});
  const int64_t pblocks =
      std::max<int64_t>(1, std::min<int64_t>((work + kBlock - 1) / kBlock, 4 * int64_t(h->n_cu)));
  hipLaunchKernelGGL(k_prep, dim3(unsigned(pblocks)), dim3(kBlock), 0, s, p);
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? ARCHEAD_OK : hip_fail(e, "prologue launch");
}

// MFMA path prologue: the head-derived tables (unless the head has them
// prepared), then stage 1 (t and the group biases).
archead_status launch_mfma_prologue(const archead_handle* h, const void* x, int64_t M,
                                    int64_t ldx, const WsLayout& w, char* ws, hipStream_t s) {
  const archead_desc& d = h->desc;
  const int R = int(d.r_c + d.r_r);
  const int nch_u = exp_chunks(d.r_c), nch = nch_u + exp_chunks(d.r_r);
  const int nslot = int(d.d / d.g) + (d.r_c ? 1 : 0) + (d.r_r ? 1 : 0);
  char* pb = prep_base(h, w, ws);
  if (!h->prep.load(std::memory_order_acquire)) {
    archead_status st = launch_prep(h, pb, s);
    if (st != ARCHEAD_OK) return st;
  }
  Stage1MArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.ldx = ldx; a.M = M; a.d = int(d.d); a.g = int(d.g);
  a.wbf = reinterpret_cast<const uint16_t*>(pb + prep_layout(h).wbf_off);
  a.sv = static_cast<const uint16_t*>(h->ptrs.core_v_scale);
  a.gv = int(d.r_c ? d.g_v : d.d); a.rc = int(d.r_c);
  a.sb = static_cast<const uint16_t*>(h->ptrs.corr_b_scale);
  a.gb = int(d.r_r ? d.g_b : d.d); a.rr = int(d.r_r);
  a.tsplit = reinterpret_cast<uint16_t*>(ws + w.ts_off);
  a.nch = nch; a.nch_u = nch_u;
  a.gbias = reinterpret_cast<float*>(ws + w.gb_off);
  a.nslot = nslot;
  a.ksplit = s1_ksplit(h, M);
  a.tpart = reinterpret_cast<float*>(ws + w.s1p_off);
  const int64_t mblocks = (M + kS1MTok - 1) / kS1MTok;
  const int64_t rblocks = R > 0 ? (R + kS1MCols - 1) / kS1MCols : 1;
  if (mblocks > 0x7fffffff) return fail(ARCHEAD_E_UNSUPPORTED, "M too large");
  hipLaunchKernelGGL(k_stage1m, dim3(unsigned(mblocks), unsigned(rblocks), unsigned(a.ksplit)),
                     dim3(kS1MBlock), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess && a.ksplit > 1) {
    const int64_t n = M * R;
    hipLaunchKernelGGL(k_stage1m_fin, dim3(unsigned((n + kBlock - 1) / kBlock)), dim3(kBlock), 0,
                       s, a);
    e = hipGetLastError();
  }
  return e == hipSuccess ? ARCHEAD_OK : hip_fail(e, "stage-1 launch");
}

// Call stamp of the decode kernels' stage-1 exchange: unique per call
// within the process (the low bits count calls, the start value is drawn
// from the clock so stamps left in reused memory by another process are
// unlikely to match).
uint32_t next_epoch() {
  static std::atomic<uint32_t> counter{uint32_t(
      std::chrono::steady_clock::now().time_since_epoch().count() * 2654435761ull)};
  return counter.fetch_add(1, std::memory_order_relaxed) + 1u;
}

// Stage-1 operands of a call (V_c, B_w and their scales, the stamped t in
// the workspace, a fresh epoch).
Stage1Ops stage1_ops(const archead_handle* h, uint64_t* tst) {
  const archead_desc& d = h->desc;
  Stage1Ops o;
  o.cv = static_cast<const int8_t*>(h->ptrs.core_v);
  o.sv = static_cast<const uint16_t*>(h->ptrs.core_v_scale);
  o.cb = static_cast<const int8_t*>(h->ptrs.corr_b);
  o.sb = static_cast<const uint16_t*>(h->ptrs.corr_b_scale);
  o.gv = int(d.r_c ? d.g_v : d.d);
  o.gb = int(d.r_r ? d.g_b : d.d);
  o.rc = int(d.r_c);
  o.rr = int(d.r_r);
  o.d = int(d.d);
  o.tst = reinterpret_cast<unsigned long long*>(tst);
  o.epoch = next_epoch();
  o.spin_limit = h->t_spin_limit;
  return o;
}

GemvArgs gemv_args(const archead_handle* h, const void* x, int64_t ldx, uint64_t* tst) {
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
  a.s1 = stage1_ops(h, tst);
  a.n_prod_blocks = int((d.r_c + d.r_r + kWaves - 1) / kWaves);
  a.V = d.V; a.d = int(d.d); a.g = int(d.g); a.rc = int(d.r_c); a.rr = int(d.r_r);
  const int64_t cpg = d.g / 32;
  a.gshift = (cpg & (cpg - 1)) == 0 ? __builtin_ctzll(uint64_t(cpg)) : -1;
  const int lpr = lanes_per_row(d);
  const int kd = lpr >= 64 ? 1 : 2;   // ExpLanes<LPR>::KD
  const int64_t ngrp = d.d / d.g;
  const bool sc8 = d.scale_dtype == ARCHEAD_U8;
  // a step's scales: 2 (fp16) or 4 (8-bit codes) groups per segment lane
  const int64_t gpl = sc8 ? 4 : 2;
  a.fast = d.r_c % 4 == 0 && d.r_r % 4 == 0 && (d.r_c + d.r_r) / 4 <= int64_t(kd) * lpr &&
           (d.r_c == 0 || aligned(h->ptrs.core_u, 4)) &&
           (d.r_r == 0 || aligned(h->ptrs.corr_a, 4)) && ngrp % gpl == 0 && ngrp <= gpl * lpr;
  a.rrs = sc8 ? static_cast<const uint16_t*>(h->ptrs.res_row_scales) : a.rs;
  // an absent factor reads the (valid, 16-byte aligned) residual buffers with
  // stride 0 instead; its contribution is masked to zero in the kernel
  a.cu_stride = d.r_c; a.su_stride = d.r_c ? 1 : 0;
  a.ca_stride = d.r_r; a.sa_stride = d.r_r ? 1 : 0;
  if (!d.r_c) { a.cu = reinterpret_cast<const int8_t*>(a.codes); a.su = a.rs; }
  if (!d.r_r) { a.ca = reinterpret_cast<const int8_t*>(a.codes); a.sa = a.rs; }
  const int64_t wr = gemv_rows_per_step(d);
  a.nsteps = (d.V + wr - 1) / wr;
  a.nit = int((d.d / 32) / lanes_per_row(d));
  return a;
}

// One launch per group of up to 4 tokens.  forced_grid > 0 fixes the grid
// (the CE passes, whose partials are indexed by workgroup).
archead_status launch_gemv_passes(const archead_handle* h, GemvArgs a, int64_t M, bool ce,
                                  int64_t forced_grid, hipStream_t s) {
  const int lpr = lanes_per_row(h->desc);
  // timing events (if set) are attached to the first and last dispatch
  // packets themselves, so they bracket exactly the kernel execution
  hipEvent_t ev0 = static_cast<hipEvent_t>(h->ev_start.load(std::memory_order_relaxed));
  hipEvent_t ev1 = static_cast<hipEvent_t>(h->ev_stop.load(std::memory_order_relaxed));
  for (int64_t m0 = 0; m0 < M; m0 += 4) {
    const int tok = int(M - m0 < 4 ? M - m0 : 4);
    const bool sc8 = h->desc.scale_dtype == ARCHEAD_U8;
    GemvFn fn = ce ? gemv_fn<true>(tok, lpr, sc8) : gemv_fn<false>(tok, lpr, sc8);
    const int64_t grid = a.n_prod_blocks + (forced_grid > 0 ? forced_grid : gemv_grid(h, tok, ce));
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

using DecFn = void (*)(DecArgs);

template <bool CE, int EK, bool SC8>
DecFn dec_fn_ek(int gw) {
  switch (gw) {
    case 1: return k_dec<1, CE, EK, SC8>;
    case 2: return k_dec<2, CE, EK, SC8>;
    default: return k_dec<4, CE, EK, SC8>;
  }
}

template <bool CE, bool SC8>
DecFn dec_fn_sc(int gw, int kcu, int kca) {
  return kcu <= 2 && kca <= 2 ? dec_fn_ek<CE, 2, SC8>(gw) : dec_fn_ek<CE, 4, SC8>(gw);
}

template <bool CE>
DecFn dec_fn(int gw, int kcu, int kca, bool sc8) {
  return sc8 ? dec_fn_sc<CE, true>(gw, kcu, kca) : dec_fn_sc<CE, false>(gw, kcu, kca);
}

// One launch per pass of up to dec_tokens_per_pass tokens.  The CE form
// writes one softmax partial per consumer workgroup.
archead_status launch_dec(const archead_handle* h, const void* x, int64_t M, int64_t ldx,
                          uint64_t* tst, DecArgs a, bool ce, hipStream_t s) {
  const archead_desc& d = h->desc;
  const DecGrid gr = dec_grid(h);
  const int tpp = dec_tokens_per_pass(d);
  a.codes = static_cast<const uint8_t*>(h->ptrs.res_codes);
  a.rs = static_cast<const uint16_t*>(h->ptrs.res_scales);
  a.cu = static_cast<const int8_t*>(h->ptrs.core_u);
  a.su = static_cast<const uint16_t*>(h->ptrs.core_u_scale);
  a.ca = static_cast<const int8_t*>(h->ptrs.corr_a);
  a.sa = static_cast<const uint16_t*>(h->ptrs.corr_a_scale);
  a.s1 = stage1_ops(h, tst);
  a.x = static_cast<const uint16_t*>(x);
  a.ldx = ldx;
  a.V = d.V;
  a.d = int(d.d); a.g = int(d.g); a.rc = int(d.r_c); a.rr = int(d.r_r);
  a.ngrp = int(d.d / d.g);
  a.n_units = gr.n_units;
  a.n_waves = gr.n_waves;
  a.n_prod_blocks = gr.prod_blocks;
  const int gw = int(d.g / 32);
  const DecLds l0 = dec_lds(d, 1);
  const bool sc8 = d.scale_dtype == ARCHEAD_U8;
  DecFn fn = ce ? dec_fn<true>(gw, l0.kcu, l0.kca, sc8) : dec_fn<false>(gw, l0.kcu, l0.kca, sc8);
  a.rrs = sc8 ? static_cast<const uint16_t*>(h->ptrs.res_row_scales) : a.rs;
  hipEvent_t ev0 = static_cast<hipEvent_t>(h->ev_start.load(std::memory_order_relaxed));
  hipEvent_t ev1 = static_cast<hipEvent_t>(h->ev_stop.load(std::memory_order_relaxed));
  const int64_t grid = gr.prod_blocks + gr.consumer_blocks;
  for (int64_t m0 = 0; m0 < M; m0 += tpp) {
    const int tok = int(M - m0 < tpp ? M - m0 : tpp);
    const DecLds l = dec_lds(d, tok);
    a.tok0 = m0;
    a.M = tok;
    a.kcu = l.kcu; a.kca = l.kca;
    a.xstr = l.xstr; a.tstr = l.tstr;
    a.off_bias = l.off_bias; a.off_t = l.off_t; a.off_red = l.off_red;
    if (l.total > 65536) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, l.total);
      if (e != hipSuccess) return hip_fail(e, "decode LDS size attribute");
    }
    void* args[] = {&a};
    const bool first = m0 == 0, last = m0 + tpp >= M;
    hipError_t e = hipExtLaunchKernel(reinterpret_cast<const void*>(fn), dim3(unsigned(grid)),
                                      dim3(kDBlock), args, size_t(l.total), s,
                                      first ? ev0 : nullptr, last ? ev1 : nullptr, 0);
    if (e != hipSuccess) return hip_fail(e, "MFMA decode launch");
  }
  return ARCHEAD_OK;
}

using MidFn = void (*)(MidArgs);

// Tiles of 32 tokens (two MFMA row blocks) and 3 units per wave (groups of
// 128) or 2 (groups of 64): the largest that keep the main loop within the
// register budget.  (Tiles of 64 tokens with 2 units per wave measured
// slower than two tiles of 32.)
template <bool CE>
MidFn mid_fn(int gw, bool sc8) {
  if (sc8) return gw == 4 ? k_mid<4, 2, 3, CE, true> : k_mid<2, 2, 2, CE, true>;
  return gw == 4 ? k_mid<4, 2, 3, CE, false> : k_mid<2, 2, 2, CE, false>;
}

// One launch per tile of up to 32 tokens.  The CE form writes one softmax
// partial per consumer workgroup.
archead_status launch_mid(const archead_handle* h, const void* x, int64_t M, int64_t ldx,
                          uint64_t* tst, MidArgs a, bool ce, hipStream_t s) {
  const archead_desc& d = h->desc;
  const MidGrid gr = mid_grid(h);
  a.codes = static_cast<const uint8_t*>(h->ptrs.res_codes);
  a.rs = static_cast<const uint16_t*>(h->ptrs.res_scales);
  a.rrs = d.scale_dtype == ARCHEAD_U8 ? static_cast<const uint16_t*>(h->ptrs.res_row_scales) : a.rs;
  a.cu = static_cast<const int8_t*>(h->ptrs.core_u);
  a.su = static_cast<const uint16_t*>(h->ptrs.core_u_scale);
  a.ca = static_cast<const int8_t*>(h->ptrs.corr_a);
  a.sa = static_cast<const uint16_t*>(h->ptrs.corr_a_scale);
  a.s1 = stage1_ops(h, tst);
  a.x = static_cast<const uint16_t*>(x);
  a.ldx = ldx;
  a.V = d.V;
  a.d = int(d.d); a.rc = int(d.r_c); a.rr = int(d.r_r);
  a.ngrp = int(d.d / d.g);
  a.n_units = gr.n_units;
  a.n_cblocks = int(gr.cblocks);
  a.n_prod_blocks = gr.prod_blocks;
  const int gw = int(d.g / 32);
  hipEvent_t ev0 = static_cast<hipEvent_t>(h->ev_start.load(std::memory_order_relaxed));
  hipEvent_t ev1 = static_cast<hipEvent_t>(h->ev_stop.load(std::memory_order_relaxed));
  const int64_t grid = gr.prod_blocks + gr.cblocks;
  for (int64_t m0 = 0; m0 < M; m0 += kMidTokMax) {
    const int tok = int(M - m0 < kMidTokMax ? M - m0 : kMidTokMax);
    const bool sc8 = d.scale_dtype == ARCHEAD_U8;
    MidFn fn = ce ? mid_fn<true>(gw, sc8) : mid_fn<false>(gw, sc8);
    const MidLds l = mid_lds(d);
    a.tok0 = m0;
    a.M = tok;
    a.kcu = l.kcu; a.kca = l.kca;
    a.tstr = l.tstr;
    a.off_bias = l.off_bias; a.off_red = l.off_red; a.off_y = l.off_y; a.off_idx = l.off_idx;
    a.off_sc = l.off_sc;
    if (l.total > 65536) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, l.total);
      if (e != hipSuccess) return hip_fail(e, "several-token LDS size attribute");
    }
    void* args[] = {&a};
    const bool first = m0 == 0, last = m0 + kMidTokMax >= M;
    hipError_t e = hipExtLaunchKernel(reinterpret_cast<const void*>(fn), dim3(unsigned(grid)),
                                      dim3(kMidBlock), args, size_t(l.total), s,
                                      first ? ev0 : nullptr, last ? ev1 : nullptr, 0);
    if (e != hipSuccess) return hip_fail(e, "several-token launch");
  }
  return ARCHEAD_OK;
}

MfmaArgs mfma_args(const archead_handle* h, const void* x, int64_t M, int64_t ldx,
                   const WsLayout& w, char* ws) {
  const archead_desc& d = h->desc;
  MfmaArgs a;
  memset(&a, 0, sizeof a);
  a.codes = static_cast<const uint8_t*>(h->ptrs.res_codes);
  a.x = static_cast<const uint16_t*>(x);
  a.ldx = ldx;
  a.tsplit = reinterpret_cast<const uint16_t*>(ws + w.ts_off);
  const PrepLayout pl = prep_layout(h);
  const char* pb = prep_base(h, w, ws);
  a.ucodes = reinterpret_cast<const int8_t*>(pb + pl.uc_off);
  a.gbias = reinterpret_cast<const float*>(ws + w.gb_off);
  a.ratio = reinterpret_cast<const float*>(pb + pl.rat_off);
  a.fin = reinterpret_cast<const float*>(pb + pl.fin_off);
  a.M = M; a.V = d.V;
  a.d = int(d.d); a.g = int(d.g);
  a.nslot = int(d.d / d.g) + (d.r_c ? 1 : 0) + (d.r_r ? 1 : 0);
  a.nch_u = exp_chunks(d.r_c);
  a.nch = a.nch_u + exp_chunks(d.r_r);
  a.n_mt = (M + kTM - 1) / kTM;
  a.n_vt = (d.V + kTN - 1) / kTN;
  a.n_tiles = a.n_vt * a.n_mt;
  a.tiles_per_xcd = (a.n_tiles + 7) / 8;
  return a;
}

archead_status launch_mfma(const archead_handle* h, MfmaArgs& a, bool ce, hipStream_t s) {
  // byte ranges of one tile's buffers must stay below 2 GiB
  if (int64_t(kTM) * a.ldx * 2 >= (int64_t(1) << 31))
    return fail(ARCHEAD_E_UNSUPPORTED, "ldx too large for the many-token kernel");
  const void* fn = ce ? reinterpret_cast<const void*>(k_mfma<true>)
                      : reinterpret_cast<const void*>(k_mfma<false>);
  const int lds = MGeom::LDS;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return hip_fail(e, "MFMA LDS size attribute");
  hipEvent_t ev0 = static_cast<hipEvent_t>(h->ev_start.load(std::memory_order_relaxed));
  hipEvent_t ev1 = static_cast<hipEvent_t>(h->ev_stop.load(std::memory_order_relaxed));
  void* args[] = {&a};
  const int64_t grid = 8 * a.tiles_per_xcd;
  if (grid > 0x7fffffff) return fail(ARCHEAD_E_UNSUPPORTED, "too many MFMA tiles");
  e = hipExtLaunchKernel(fn, dim3(unsigned(grid)), dim3(kMBlock), args, size_t(lds), s, ev0, ev1, 0);
  return e == hipSuccess ? ARCHEAD_OK : hip_fail(e, "MFMA launch");
}

// The fused-softmax pass of every kernel: per token and partial (a
// workgroup, or a vocabulary tile) the (max, sum exp) pair, the target's
// logit when targets is not null, and the argmax partials when pidx is not
// null.
archead_status launch_softmax_partials(const archead_handle* h, const void* x, int64_t M,
                                       int64_t ldx, const void* targets, bool tgt64,
                                       const WsLayout& w, char* base, int* pidx, hipStream_t s) {
  float2* part = reinterpret_cast<float2*>(base + w.part_off);
  float* tl = reinterpret_cast<float*>(base + w.tgt_off);
  const int64_t n_part = w.n_part;
  const Path path = choose_path(h, M);
  if (path == Path::kDec) {
    DecArgs a;
    memset(&a, 0, sizeof a);
    a.tgt = targets;
    a.tgt64 = tgt64;
    a.part = part;
    a.part_idx = pidx;
    a.n_part = n_part;
    a.tgt_logit = tl;
    return launch_dec(h, x, M, ldx, reinterpret_cast<uint64_t*>(base + w.tst_off), a, true, s);
  }
  if (path == Path::kMid) {
    MidArgs a;
    memset(&a, 0, sizeof a);
    a.tgt = targets;
    a.tgt64 = tgt64;
    a.part = part;
    a.part_idx = pidx;
    a.n_part = n_part;
    a.tgt_logit = tl;
    return launch_mid(h, x, M, ldx, reinterpret_cast<uint64_t*>(base + w.tst_off), a, true, s);
  }
  if (path == Path::kTiled) {
    archead_status st = launch_mfma_prologue(h, x, M, ldx, w, base, s);
    if (st != ARCHEAD_OK) return st;
    MfmaArgs a = mfma_args(h, x, M, ldx, w, base);
    a.tgt = targets;
    a.tgt64 = tgt64;
    a.part = part;
    a.part_idx = pidx;
    a.tgt_logit = tl;
    return launch_mfma(h, a, true, s);
  }
  GemvArgs a = gemv_args(h, x, ldx, reinterpret_cast<uint64_t*>(base + w.tst_off));
  a.tgt = targets;
  a.tgt64 = tgt64;
  a.part = part;
  a.part_idx = pidx;
  a.n_part = n_part;
  a.tgt_logit = tl;
  return launch_gemv_passes(h, a, M, true, n_part, s);
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
  if (d.scale_dtype == ARCHEAD_U8 && (!ptrs->res_row_scales || !aligned(ptrs->res_row_scales, 2)))
    return fail(ARCHEAD_E_INVALID_ARG,
                "8-bit scale codes need res_row_scales (fp16 [V], 2-byte aligned)");
  if (d.r_c && (!ptrs->core_u || !ptrs->core_u_scale || !ptrs->core_v || !ptrs->core_v_scale))
    return fail(ARCHEAD_E_INVALID_ARG, "r_c > 0 needs core_u, core_u_scale, core_v, core_v_scale");
  if (d.r_r && (!ptrs->corr_a || !ptrs->corr_a_scale || !ptrs->corr_b || !ptrs->corr_b_scale))
    return fail(ARCHEAD_E_INVALID_ARG, "r_r > 0 needs corr_a, corr_a_scale, corr_b, corr_b_scale");
  if (!aligned(ptrs->res_codes, 16)) return fail(ARCHEAD_E_MISALIGNED, "res_codes must be 16-byte aligned");
  const void* f16s[] = {d.scale_dtype == ARCHEAD_F16 ? ptrs->res_scales : nullptr,
                        ptrs->core_u_scale, ptrs->core_v_scale, ptrs->corr_a_scale,
                        ptrs->corr_b_scale};
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
  st = scratch_setup(dev);
  if (st != ARCHEAD_OK) return st;
  archead_handle* h = new (std::nothrow) archead_handle();
  if (!h) return fail(ARCHEAD_E_INVALID_ARG, "out of host memory");
  h->desc = d;
  h->ptrs = *ptrs;
  h->device = dev;
  h->n_cu = prop.multiProcessorCount;
  h->gemv_max_m.store(kDefaultGemvMaxM);
  {
    int64_t r[4];
    default_ranges(d, r);
    h->dec_min_m.store(r[0]);
    h->dec_max_m.store(r[1]);
    h->mid_min_m.store(r[2]);
    h->mid_max_m.store(r[3]);
  }
  // polls of the stage-1 exchange before the fallback (ARCHEAD_T_SPIN_LIMIT
  // overrides; 0 makes every value take the fallback, for its tests)
  h->t_spin_limit = 1 << 16;
  if (const char* e = getenv("ARCHEAD_T_SPIN_LIMIT")) h->t_spin_limit = atoi(e) >= 0 ? atoi(e) : h->t_spin_limit;
  for (auto& c : h->grid_cache) c.store(0);
  h->ev_start.store(nullptr);
  h->ev_stop.store(nullptr);
  h->prep.store(nullptr);
  *out = h;
  return ARCHEAD_OK;
}

void archead_destroy(archead_handle* h) { delete h; }

size_t archead_workspace_bytes(const archead_handle* h, int64_t M, archead_op op) {
  if (!h || M <= 0) return 0;
  return ws_layout(h, M, op).total;
}

size_t archead_prepared_bytes(const archead_handle* h) {
  if (!h || !mfma_ok(h)) return 0;
  return prep_layout(h).total;
}

archead_status archead_prepare(archead_handle* h, void* buf, size_t bytes, void* stream) {
  clear_error();
  if (!h) return fail(ARCHEAD_E_INVALID_ARG, "handle is NULL");
  if (!buf) {
    if (bytes) return fail(ARCHEAD_E_INVALID_ARG, "buf is NULL with bytes > 0");
    h->prep.store(nullptr, std::memory_order_release);
    return ARCHEAD_OK;
  }
  if (!mfma_ok(h)) return fail(ARCHEAD_E_UNSUPPORTED, "the head shape has no many-token kernel");
  if (!aligned(buf, 256)) return fail(ARCHEAD_E_MISALIGNED, "buf must be 256-byte aligned");
  const size_t need = prep_layout(h).total;
  if (bytes < need) return fail(ARCHEAD_E_WORKSPACE, "buffer %zu < %zu bytes", bytes, need);
  h->prep.store(nullptr, std::memory_order_release);
  archead_status st = launch_prep(h, static_cast<char*>(buf), static_cast<hipStream_t>(stream));
  if (st != ARCHEAD_OK) return st;
  h->prep.store(static_cast<char*>(buf), std::memory_order_release);
  return ARCHEAD_OK;
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
  const Path path = choose_path(h, M);
  if (path == Path::kDec) {
    DecArgs a;
    memset(&a, 0, sizeof a);
    a.out = out;
    a.ldo = ldo;
    a.out_bf16 = out_dtype == ARCHEAD_BF16;
    return launch_dec(h, x, M, ldx,
                      reinterpret_cast<uint64_t*>(static_cast<char*>(ws) + w.tst_off), a, false,
                      s);
  }
  if (path == Path::kMid) {
    MidArgs a;
    memset(&a, 0, sizeof a);
    a.out = out;
    a.ldo = ldo;
    a.out_bf16 = out_dtype == ARCHEAD_BF16;
    return launch_mid(h, x, M, ldx,
                      reinterpret_cast<uint64_t*>(static_cast<char*>(ws) + w.tst_off), a, false,
                      s);
  }
  if (path == Path::kTiled) {
    st = launch_mfma_prologue(h, x, M, ldx, w, static_cast<char*>(ws), s);
    if (st != ARCHEAD_OK) return st;
    MfmaArgs a = mfma_args(h, x, M, ldx, w, static_cast<char*>(ws));
    a.out = out;
    a.ldo = ldo;
    a.out_bf16 = out_dtype == ARCHEAD_BF16;
    return launch_mfma(h, a, false, s);
  }
  GemvArgs a = gemv_args(h, x, ldx, reinterpret_cast<uint64_t*>(static_cast<char*>(ws) + w.tst_off));
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
  st = launch_softmax_partials(h, x, M, ldx, targets, tgt_dtype == ARCHEAD_I64, w,
                               static_cast<char*>(ws), nullptr, s);
  if (st != ARCHEAD_OK) return st;
  char* base = static_cast<char*>(ws);
  const float2* part = reinterpret_cast<const float2*>(base + w.part_off);
  const float* tl = reinterpret_cast<const float*>(base + w.tgt_off);
  hipLaunchKernelGGL(k_ce_merge, dim3(unsigned(M)), dim3(kBlock), 0, s, part, w.n_part, targets,
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

archead_status archead_logits_argmax(const archead_handle* h, const void* x, int64_t M,
                                     int64_t ldx, int64_t* idx, float* max_logit, void* ws,
                                     size_t ws_bytes, void* stream) {
  clear_error();
  archead_status st = check_call(h, x, M, ldx, ws, ws_bytes, ARCHEAD_OP_ARGMAX);
  if (st != ARCHEAD_OK || M == 0) return st;
  if (!idx) return fail(ARCHEAD_E_INVALID_ARG, "idx is required");
  if (!aligned(idx, 8) || (max_logit && !aligned(max_logit, 4)))
    return fail(ARCHEAD_E_MISALIGNED, "idx / max_logit misaligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const WsLayout w = ws_layout(h, M, ARCHEAD_OP_ARGMAX);
  char* base = static_cast<char*>(ws);
  int* pidx = reinterpret_cast<int*>(base + w.pidx_off);
  st = launch_softmax_partials(h, x, M, ldx, nullptr, false, w, base, pidx, s);
  if (st != ARCHEAD_OK) return st;
  const float2* part = reinterpret_cast<const float2*>(base + w.part_off);
  hipLaunchKernelGGL(k_argmax_merge, dim3(unsigned(M)), dim3(kBlock), 0, s, part, pidx,
                     w.n_part, idx, max_logit);
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? ARCHEAD_OK : hip_fail(e, "argmax merge launch");
}

}  // extern "C"
