// Device helpers shared by the kernels of the packed-head forward: vector
// types, loads, the INT4 unpack, bf16 conversions, the softmax merge, the
// in-launch stage 1 (t = x V_c^T, x B_w^T), MFMA fragment helpers.
#pragma once

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
// A GEMV step is 8 rows per lane segment with 1 iteration of loads in flight
// (steps of 2 or 4 rows with the same bytes in flight measured slower: the
// shorter last round of the grid does not repay the per-step work).
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

// ----------------------------------------- factor codes of U_c and A_w
// The rank-r expansion reads the codes of its vocabulary rows.  Heads whose
// ranks are multiples of 4 with int8 codes are read as aligned dwords by the
// kernels themselves; the helpers below serve every other head ("general"
// factor codes): ranks of any size, and the core-left codes as ARCHEAD_I5
// words (six 5-bit two's complement fields per little-endian 32-bit word,
// field k % 6 of word k / 6 at bits 5 (k % 6)).

// field j (0..5) of an ARCHEAD_I5 word, sign-extended
__device__ __forceinline__ int i5_field(uint32_t w, int j) { return int(w << (27 - 5 * j)) >> 27; }

// Eight codes k0 .. k0 + 7 (k0 % 8 == 0) of the row starting at byte `row`
// of a buffer resource, as int8 in two little-endian dwords: from ARCHEAD_I5
// words (U5; rows of 4 ceil(r/6) bytes: two aligned word loads), or from int8
// codes at any byte offset (three aligned dword loads joined with
// v_alignbyte).  No branch, so the loads of the stream in flight are not
// drained.  Codes at or past the rank are finite but unspecified (the
// kernels pair them with zero t); reads past the resource come back as zero.
template <bool U5>
__device__ __forceinline__ u32x2_t fcodes8(__amdgpu_buffer_rsrc_t r, int row, int k0) {
  if constexpr (U5) {
    const int w = k0 / 6;
    const uint32_t w0 = __builtin_amdgcn_raw_buffer_load_b32(r, row + 4 * w, 0, 0);
    const uint32_t w1 = __builtin_amdgcn_raw_buffer_load_b32(r, row + 4 * w + 4, 0, 0);
    const int j0 = k0 - 6 * w;
    uint32_t o[2] = {0u, 0u};
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int j = j0 + i;
      const int c = j < 6 ? i5_field(w0, j) : i5_field(w1, j - 6);
      o[i >> 2] |= (uint32_t(c) & 0xffu) << (8 * (i & 3));
    }
    return u32x2_t{o[0], o[1]};
  } else {
    const int off = row + k0, al = off & ~3;
    const uint32_t w0 = __builtin_amdgcn_raw_buffer_load_b32(r, al, 0, 0);
    const uint32_t w1 = __builtin_amdgcn_raw_buffer_load_b32(r, al + 4, 0, 0);
    const uint32_t w2 = __builtin_amdgcn_raw_buffer_load_b32(r, al + 8, 0, 0);
    const uint32_t sh = uint32_t(off & 3);
    return u32x2_t{__builtin_amdgcn_alignbyte(w1, w0, sh), __builtin_amdgcn_alignbyte(w2, w1, sh)};
  }
}

// Four codes k0 .. k0 + 3 (k0 % 4 == 0) of the row starting at byte `row` of
// a buffer resource, as int8 in one little-endian dword, likewise (two
// aligned loads in both formats).
template <bool U5>
__device__ __forceinline__ uint32_t fcodes4(__amdgpu_buffer_rsrc_t r, int row, int k0) {
  if constexpr (U5) {
    const int w = k0 / 6;
    const uint32_t w0 = __builtin_amdgcn_raw_buffer_load_b32(r, row + 4 * w, 0, 0);
    const uint32_t w1 = __builtin_amdgcn_raw_buffer_load_b32(r, row + 4 * w + 4, 0, 0);
    uint32_t o = 0u;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = k0 + i - 6 * w;
      const int c = j < 6 ? i5_field(w0, j) : i5_field(w1, j - 6);
      o |= (uint32_t(c) & 0xffu) << (8 * i);
    }
    return o;
  } else {
    const int off = row + k0, al = off & ~3;
    const uint32_t w0 = __builtin_amdgcn_raw_buffer_load_b32(r, al, 0, 0);
    const uint32_t w1 = __builtin_amdgcn_raw_buffer_load_b32(r, al + 4, 0, 0);
    return __builtin_amdgcn_alignbyte(w1, w0, uint32_t(off & 3));
  }
}

// fcodes4 in two halves, so the loads stay in flight until the codes are
// used: fcodes4_fetch requests the two aligned words, fcodes4_decode joins
// them later (int8 codes: sh = the byte offset of the first code, (row + k0)
// & 3, which the caller recomputes from the row).
struct RawCodes4 {
  uint32_t w0, w1;
};
template <bool U5>
__device__ __forceinline__ RawCodes4 fcodes4_fetch(__amdgpu_buffer_rsrc_t r, int row, int k0) {
  RawCodes4 c;
  if constexpr (U5) {
    const int w = k0 / 6;
    c.w0 = __builtin_amdgcn_raw_buffer_load_b32(r, row + 4 * w, 0, 0);
    c.w1 = __builtin_amdgcn_raw_buffer_load_b32(r, row + 4 * w + 4, 0, 0);
  } else {
    const int al = (row + k0) & ~3;
    c.w0 = __builtin_amdgcn_raw_buffer_load_b32(r, al, 0, 0);
    c.w1 = __builtin_amdgcn_raw_buffer_load_b32(r, al + 4, 0, 0);
  }
  return c;
}
template <bool U5>
__device__ __forceinline__ uint32_t fcodes4_decode(const RawCodes4& c, int k0, uint32_t sh) {
  if constexpr (U5) {
    const int w = k0 / 6;
    uint32_t o = 0u;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int j = k0 + i - 6 * w;
      const int v = j < 6 ? i5_field(c.w0, j) : i5_field(c.w1, j - 6);
      o |= (uint32_t(v) & 0xffu) << (8 * i);
    }
    return o;
  } else {
    return __builtin_amdgcn_alignbyte(c.w1, c.w0, sh);
  }
}

// code k of a row (rowp: its first byte), int8 or ARCHEAD_I5
__device__ __forceinline__ int fcode1(const uint8_t* rowp, int k, bool u5) {
  if (u5) return i5_field(reinterpret_cast<const uint32_t*>(rowp)[k / 6], k % 6);
  return int(int8_t(rowp[k]));
}

// Per-lane state of the fused epilogues (softmax, argmax, top-k).
template <int TOK>
struct CeState {
  float mx[TOK], se[TOK];
  int am[TOK];      // smallest vocabulary index attaining mx so far
  int64_t y[TOK];
  // top-k variants: this lane's slot of the wave's list and the list's bar
  float tv[TOK], bv[TOK];
  int ti[TOK], bi[TOK];
};

// "no index yet" for the argmax partials: larger than any vocabulary index
constexpr int kNoIdx = 0x7fffffff;


typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) uint8_t lds_u8;

constexpr int kTM = 256, kTN = 256;          // tile: tokens x vocabulary rows
constexpr int kMBlock = 512, kMWaves = 8;    // 2 x 4 waves of 128 x 64
constexpr int kKS = 64;                      // K elements per stage
constexpr int kRing = 3;                     // LDS stages (two loads in flight)
constexpr int kRasterGM = 4;                 // token tiles per raster group (measured: 2 and 8 slower at M = 4096)
constexpr float kZeroScale = 0x1p-60f;       // stand-in for a zero scale
constexpr int kExpDims = 16;                 // rank dimensions per expansion stage

// Geometry of the tiled kernel for TM token rows per tile and NW waves per
// workgroup: NW = 8 (2 x 4 waves of TM/2 x 64; one workgroup per CU) or
// NW = 4 (1 x 4 waves of TM x 64; TM = 128: two workgroups per CU, TM = 64:
// three), whose stage barriers are independent, so one's LDS waits, tile
// start and epilogue overlap the others' MFMAs.  A stage holds x [TM][kKS] bf16,
// codes [kTN][kKS/2], (FID: the dense head's rows [kTN][kKS] bf16,) the scale
// ratios of the kTN columns and the slot biases of the TM rows.
template <int TM, int NW = kMWaves, bool FID = false>
struct MGeomT {
  static constexpr int WMW = NW / 4;                  // waves along the tokens
  static constexpr int WM = TM / WMW;                 // token rows per wave
  static constexpr int MI = WM / 16;                  // 16-row MFMA blocks per wave
  static constexpr int XBYTES = TM * kKS * 2;         // x [TM][kKS] bf16
  static constexpr int CBYTES = kTN * kKS / 2;        // codes [kTN][kKS/2]
  static constexpr int DOFF = XBYTES + CBYTES;        // dense rows (fidelity pass)
  static constexpr int DBYTES = FID ? kTN * kKS * 2 : 0;
  static constexpr int RAT = DOFF + DBYTES;           // fp32 [kTN] scale ratios
  static constexpr int BIAS = RAT + kTN * 4;          // fp32 [TM] slot biases
  static constexpr int STAGE = BIAS + TM * 4;
  static constexpr int NX = XBYTES / 1024 / NW;       // x loads per wave and stage
  static constexpr int NC = CBYTES / 1024 / NW;       // code loads per wave and stage
  static constexpr int NA = NW == 8 ? 1 : 2;          // ratio / bias loads per wave
  static constexpr int ND = DBYTES / 1024 / NW;       // dense-row loads per wave
  static constexpr int NL = NX + NC + NA + ND;        // loads per wave and stage
  static constexpr int PPS = (NL + 2 * MI - 1) / (2 * MI);   // loads per MFMA row block
  static constexpr int LDS = kRing * STAGE;
  static constexpr int WGS = FID ? 1 : NW == 8 ? 1 : (TM == 128 ? 2 : 3);   // workgroups per CU
  static_assert(NW == 8 || (NW == 4 && (TM == 128 || TM == 64)), "layouts built");
  static_assert(!FID || (NW == 4 && TM == 64), "fidelity pass: 64-row tiles of 4 waves");
  static_assert(XBYTES % (1024 * NW) == 0 && CBYTES % (1024 * NW) == 0 &&
                DBYTES % (1024 * NW) == 0, "whole loads");
  static_assert(LDS * WGS <= 160 * 1024, "LDS budget");
  static_assert(TM % 64 == 0 && TM <= kTM, "bias loads of 64 rows per wave");
};
using MGeom = MGeomT<kTM>;

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

// ------------------------------------------------------------ top-k lists
// Calls f(integral_constant<J>) for J = I .. N-1 until one returns true.
template <int I, int N, typename F>
__device__ __forceinline__ bool unroll_until(F& f) {
  if constexpr (I < N) {
    if (f(std::integral_constant<int, I>{})) return true;
    return unroll_until<I + 1, N>(f);
  }
  return false;
}

// A wave keeps the k best (value, index) pairs it has seen as one sorted
// list spread over its lanes: lane j < k holds the j-th best, in the order
// "larger value first, equal values by smaller index" (the order of the
// first-index argmax); lanes j >= k and unfilled slots hold the empty entry
// (-inf, kNoIdx), which no entry is ranked below.  NaN values never enter.
// Every helper here is called by all 64 lanes of the wave together, with a
// wave-uniform k (1 <= k <= 64).
constexpr int kTopKMax = 64;

__device__ __forceinline__ bool tk_better(float av, int ai, float bv, int bi) {
  return (av > bv) | ((av == bv) & (ai < bi));   // non-short-circuit: no branches
}

__device__ __forceinline__ float rlane_f(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

// Insert the wave-uniform pair (cv, ci): it lands at the first slot it is
// ranked above, the entries from there on move down one lane, the k-th drops
// out.  (bv, bi), the list's k-th entry (the bar a pair must beat to enter),
// is refreshed.
__device__ __forceinline__ void tk_insert(float& lv, int& li, float& bv, int& bi, float cv,
                                          int ci, int lane, int k) {
  // the previous lane's entry: DPP wave_shr:1 (a VALU move, no LDS trip)
  const int pi = __builtin_amdgcn_update_dpp(0, li, 0x138, 0xF, 0xF, true);
  const float pv = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(lv), 0x138, 0xF, 0xF, true));
  const bool here = (lane < k) & tk_better(cv, ci, lv, li);
  const bool above = (lane > 0) & tk_better(cv, ci, pv, pi);
  lv = here ? (above ? pv : cv) : lv;
  li = here ? (above ? pi : ci) : li;
  bv = rlane_f(lv, k - 1);
  bi = __builtin_amdgcn_readlane(li, k - 1);
}

// Offer one pair per lane (taken where ok): the pairs that beat the bar
// enter one at a time, in lane order.
__device__ __forceinline__ void tk_offer(float& lv, int& li, float& bv, int& bi, float v, int i,
                                         bool ok, int lane, int k) {
  uint64_t m = __ballot(ok & tk_better(v, i, bv, bi));
  while (m) {
    const int s = __builtin_ctzll(m);
    m &= m - 1;
    const float cv = rlane_f(v, s);
    const int ci = __builtin_amdgcn_readlane(i, s);
    if (tk_better(cv, ci, bv, bi)) tk_insert(lv, li, bv, bi, cv, ci, lane, k);
  }
}

// Merge the sorted lists of a workgroup's NW waves by rank: the entry in
// lane j of wave w has j better entries in its own list and, in each other
// list, as many as a binary search finds; entries have distinct indices, so
// every one has a distinct rank, and those ranked below k land in (ov, oi)
// [k] (slots no entry reaches hold the empty entry).  sv / si: LDS of NW *
// 64 entries; ov / oi: LDS of kTopKMax.  Contains two barriers: every
// thread of the workgroup calls it.
template <int NW>
__device__ __forceinline__ void tk_rank_merge(float lv, int li, int tid, int k, float* sv, int* si,
                                              float* ov, int* oi) {
  const int lane = tid & 63, wid = tid >> 6;
  sv[tid] = lv;
  si[tid] = li;
  if (tid < kTopKMax) {
    ov[tid] = -INFINITY;
    oi[tid] = kNoIdx;
  }
  __syncthreads();
  if (lane < k && li != kNoIdx) {
    int rank = lane;
    int top = 1;
    while (top * 2 <= k) top *= 2;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      if (w == wid) continue;
      const float* lw = sv + w * 64;
      const int* iw = si + w * 64;
      int pos = 0;
      for (int step = top; step > 0; step >>= 1)
        if (pos + step <= k && tk_better(lw[pos + step - 1], iw[pos + step - 1], lv, li)) pos += step;
      rank += pos;
    }
    if (rank < k) {
      ov[rank] = lv;
      oi[rank] = li;
    }
  }
  __syncthreads();
}

// Merge the lists of a workgroup's NW waves into wave 0's (the other waves'
// lists are inserted in wave order; each is sorted, so its first entry
// that fails the bar ends it).  sv / si: LDS of NW * 64 entries.  Contains
// a barrier: every wave of the workgroup calls it.
template <int NW>
__device__ __forceinline__ void tk_block_merge(float& lv, int& li, float& bv, int& bi, int lane,
                                               int wid, int k, float* sv, int* si) {
  sv[wid * 64 + lane] = lv;
  si[wid * 64 + lane] = li;
  __syncthreads();
  if (wid == 0) {
    for (int w = 1; w < NW; ++w)
      for (int j = 0; j < k; ++j) {
        const float cv = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(sv[w * 64 + j])));
        const int ci = __builtin_amdgcn_readfirstlane(si[w * 64 + j]);
        if (!tk_better(cv, ci, bv, bi)) break;
        tk_insert(lv, li, bv, bi, cv, ci, lane, k);
      }
  }
}


}  // namespace
