// The several-token kernel template (k_mid).
#pragma once

#include "dev_dec.cuh"

namespace {

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
// in steps of 128 codes of every row (lane (j, q): row j of the unit, the 16
// bytes from 16 q of the step) for all NU units at once, a 128-byte line of
// each row per request round, one line ahead; a group's partial starts from
// its bias (MFMA C input) and is scaled into the unit's total (groups of 64:
// the two groups of a step each take the step's MFMAs with the other
// group's lanes zeroed).  After the last window of a pass the window
// buffers hold t (three bf16 parts) for the rank-r expansion, then the
// units' logits go out.
// Stage 1 (t) runs in the same launch as in k_dec.
constexpr int kMidBlock = 512, kMidWaves = kMidBlock / 64;
constexpr int kMidKW = 256;   // elements of d per x window
constexpr int kMidCpol = 2;   // code loads non-temporal (read once per tile; 14% faster at 32 tokens)
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
  int cu_row;            // bytes per row of U_c (r_c int8 codes, or ARCHEAD_I5 words)
  int u5;                // U_c codes are ARCHEAD_I5 words
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

// GEN: factor-code reads as in k_dec (0 aligned int8, 1 int8 of any rank
// through fcodes8, 2 the same with ARCHEAD_I5 core-left codes).
template <int GW, int NF, int NU, bool CE, bool SC8, int GEN>
__global__ __launch_bounds__(kMidBlock) __attribute__((amdgpu_waves_per_eu(2)))
void k_mid(MidArgs a) {
  static_assert(GW == 2 || GW == 4, "groups of 64 or 128 codes");
  constexpr int TM = 16 * NF;
  constexpr int G = 32 * GW;                  // group size
  constexpr int SPW = kMidKW / G;             // groups per window
  // The head is walked in steps of 128 codes of every row: one group of
  // 128, or a pair of groups of 64 (PG groups per step, one MFMA chain and
  // scale each), so both group sizes share one loop shape and register
  // budget.  Code loads go out a 128-byte line of each row at a time (LG
  // steps: both halves of a line are requested together, not a step
  // apart), one line ahead, so the ring holds two lines of steps
  constexpr int PG = 128 / G;                 // groups per step
  constexpr int SPS = kMidKW / 128;           // steps per window
  constexpr int LG = 2;
  constexpr int NB = 2 * LG;
  static_assert((2 * SPS) % NB == 0, "ring slots are compile-time per step");
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
  const int voff_c = int(uint32_t(lr) * rowbytes) + 16 * q;   // codes: row lr, part q of a step
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
      // every lane of the group ends with the same sum (each swap adds a
      // pair of lanes' values in either order), so all of them store it:
      // no branch splits the main loop here
      sm = GW == 4 ? row16_sum(sm) : row8_sum(sm);
      bb[(c16 / (4 * GW)) * TM + row] = -float(archead::kInt4Bias) * sm;
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

  // step s: codes 128 s .. 128 s + 127 of every row (bytes 64 s ..); lane
  // (j, q) holds words 4 q .. 4 q + 3 of the step (for groups of 64:
  // quarters 0-1 the first group of the pair, 2-3 the second)
  u32x4_t cbuf[NB][NU];
  __amdgpu_buffer_rsrc_t rcu[NU];
  auto load_step = [&](auto SLOT, int s) {
    constexpr int slot = decltype(SLOT)::value;
#pragma unroll
    for (int j = 0; j < NU; ++j)
      cbuf[slot][j] = __builtin_amdgcn_raw_buffer_load_b128(rcu[j], voff_c, s * 64, kMidCpol);
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

    // iterations of two windows (2 SPS steps): window parity and ring slot
    // of every step are compile-time constants
    constexpr int IT = 2 * SPS;
    const int nstep = ngrp / PG;
#pragma unroll 1
    for (int it = 0; it < nstep / IT; ++it) {
      auto body = [&](auto J) {
        constexpr int j = decltype(J)::value;
        constexpr int par = j / SPS;             // window parity (set of its fetch)
        const int s = IT * it + j;               // this step
        const int w = 2 * it + par;              // its window
        if constexpr (j % SPS == 0) load_win(std::integral_constant<int, par>{}, w + 2);
        if constexpr (j % LG == 0) {
          // the next line of every row: steps s + LG .. s + 2 LG - 1
          auto next = [&](auto E) {
            constexpr int e = decltype(E)::value;
            const int sn = s + LG + e;
            load_step(std::integral_constant<int, (j + LG + e) % NB>{}, sn < nstep ? sn : nstep - 1);
          };
          next(std::integral_constant<int, 0>{});
          next(std::integral_constant<int, 1>{});
        }
        asm volatile("" ::: "memory");
        // four K-chunks of 32 codes per step, MFMA kc taking word kc of every
        // lane (elements 32 q + 8 kc .. of the step).  Groups of 64: each
        // group of the pair has its own chain over all four chunks, fed the
        // B fragment with the other group's quarters zeroed
        const lds_u8* const xb = L + par * (TM * kMidXstr) + (j % SPS) * 256;
        const auto* bb = sbias + par * (SPW * TM) + PG * (j % SPS) * TM;
        const uint32_t mlo = q < 2 ? 0xffffffffu : 0u;
        f32x4_t acc[PG][NU][NF];
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) {
          bf16x8_t A[NF];
#pragma unroll
          for (int f = 0; f < NF; ++f)
            A[f] = lds_load<bf16x8_t>(xb + (16 * f + lr) * kMidXstr + 16 * (4 * q + kc));
#pragma unroll
          for (int u = 0; u < NU; ++u) {
            bf16x8_t B[PG];
            if constexpr (PG == 1) {
              B[0] = unpack8(cbuf[j % NB][u][kc], kMask, kMagic);
            } else {
              const u32x4_t b = __builtin_bit_cast(u32x4_t, unpack8(cbuf[j % NB][u][kc], kMask, kMagic));
              B[0] = __builtin_bit_cast(bf16x8_t, b & mlo);
              B[PG - 1] = __builtin_bit_cast(bf16x8_t, b & ~mlo);
            }
#pragma unroll
            for (int h = 0; h < PG; ++h)
#pragma unroll
              for (int f = 0; f < NF; ++f) {
                const f32x4_t c0 =
                    kc == 0 ? *reinterpret_cast<const __attribute__((address_space(3))) f32x4_t*>(
                                  bb + h * TM + 16 * f + 4 * q)
                            : acc[h][u][f];
                acc[h][u][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[f], B[h], c0, 0, 0, 0);
              }
          }
          // one K-chunk's fragments live at a time (the scheduler would
          // otherwise hoist every chunk's LDS reads and unpacks, past the
          // register budget)
          __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int h = 0; h < PG; ++h)
#pragma unroll
          for (int u = 0; u < NU; ++u) {
            const float sc =
                f16_to_f32(lds_load<uint16_t>(ssc + (u * 16 + lr) * sstr + 2 * (PG * s + h)));
#pragma unroll
            for (int f = 0; f < NF; ++f) tot[u][f] += sc * acc[h][u][f];
          }
        if constexpr (j % SPS == SPS - 1) {
          // window w + 1 (fetched during window w - 1, or before the loop)
          store_win(std::integral_constant<int, 1 - par>{}, w + 1);
          lds_barrier();
        }
      };
      body(std::integral_constant<int, 0>{});
      body(std::integral_constant<int, 1>{});
      body(std::integral_constant<int, 2>{});
      body(std::integral_constant<int, 3>{});
    }

    // ---- rank-r expansion and the units' logits.  Its operands are
    // requested together, then t goes to LDS while they are in flight.
    u32x2_t eu[NU][4], ea[NU][4];
    uint16_t esu[NU], esa[NU];
    uint16_t ers[NU];   // row scales of 8-bit residual scale codes
#pragma unroll
    for (int j = 0; j < NU; ++j) {
      const __amdgpu_buffer_rsrc_t ru = code_rsrc(cu_b, uj[j], uint32_t(a.cu_row));
      const __amdgpu_buffer_rsrc_t ra = code_rsrc(ca_b, uj[j], uint32_t(a.rr));
#pragma unroll
      for (int kc = 0; kc < 4; ++kc) {
        if constexpr (GEN > 0) {
          // every chunk is requested (unused ones read finite codes paired
          // with zero t, or nothing past the unit), so no branch drains the
          // stream's loads
          eu[j][kc] = fcodes8<GEN == 2>(ru, lr * a.cu_row, 8 * (q * kcu + kc));
          ea[j][kc] = fcodes8<false>(ra, lr * a.rr, 8 * (q * kca + kc));
        } else {
          eu[j][kc] = __builtin_amdgcn_raw_buffer_load_b64(ru, voff_u, 8 * kc, 0);
          ea[j][kc] = __builtin_amdgcn_raw_buffer_load_b64(ra, voff_a, 8 * kc, 0);
        }
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

}  // namespace
