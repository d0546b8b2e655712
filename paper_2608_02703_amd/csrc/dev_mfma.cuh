// The tiled many-token MFMA kernel template (k_mfma) and the argument blocks
// of its prologue kernels.
#pragma once

#include "dev_common.cuh"

namespace {

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
  // logit fidelity against a dense bf16 head (XE = 1) and the rank pass (XE = 2)
  const uint16_t* dense;   // [V][ldw] bf16
  int64_t ldw;
  void* fid_part;          // [M][n_vt] FidTilePart
  const float* bref;       // [M] packed logit at the reference's top-1
  const int64_t* ref_idx;  // [M] the reference's top-1
  int64_t* rank;           // [M]
};

// One vocabulary tile's statistics of one token for the fidelity pass: the
// maxima of the dense (a) and packed (b) logits, the first index of the
// maximum of a and b there, and relative to the maxima sum e^(a - ma),
// sum e^(b - mb), sum e^(a - ma) (a - b) and sum (a - b)^2.
struct FidTilePart {
  float ma, mb, bat, sa, sb, t, sq;
  int ia;                  // vocabulary index (kNoIdx: none)
};
static_assert(sizeof(FidTilePart) == 32, "the workspace holds 32 bytes per tile and token");

// XE: 0 logits or CE (CE), 1 the fidelity pass (the dense head's rows are
// streamed through the same stages and accumulated beside the packed
// logits; per-tile FidTilePart out), 2 the rank pass (per token, packed
// logits ranked ahead of bref / ref_idx counted into rank).
// (waves per SIMD: 2 with 8-wave workgroups and with 128-row tiles of 4
// waves, two workgroups per CU; 3 with 64-row tiles, three per CU)
template <bool CE, int TM, int NW, int XE = 0>
__global__ __launch_bounds__(NW * 64)
__attribute__((amdgpu_waves_per_eu(MGeomT<TM, NW, XE == 1>::WGS * NW / 4 > 2
                                       ? MGeomT<TM, NW, XE == 1>::WGS * NW / 4 : 2)))
void k_mfma(MfmaArgs a) {
  using G = MGeomT<TM, NW, XE == 1>;
  constexpr int MI = G::MI;        // row blocks per wave
  constexpr int WM = G::WM;        // token rows per wave
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
  const int64_t m0 = mt * TM, v0 = vt * kTN;
  const int rows = int(a.M - m0 < TM ? a.M - m0 : TM);
  const int cols = int(a.V - v0 < kTN ? a.V - v0 : kTN);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = NW == 8 ? wid >> 2 : 0, wn = wid & 3;
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
  // dense rows of the tile (fidelity pass); the expansion stages load from
  // an empty resource (zeros, no memory traffic) so every stage issues the
  // same number of loads
  const uint32_t dstride = uint32_t(a.ldw) * 2;
  const __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(XE == 1 ? a.dense + v0 * a.ldw : a.x), 0,
      XE == 1 ? int((cols - 1) * dstride + uint32_t(a.d) * 2) : 0, kBufferWord3);
  const __amdgpu_buffer_rsrc_t rdz = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a.x), 0, 0, kBufferWord3);
  // auxiliary loads of this wave: the scale ratios of 64 columns and / or
  // the slot biases of 64 token rows (NW = 8: waves 0-3 the ratios, 4-7 the
  // biases; NW = 4: every wave both)
  // (the biases are laid out per 256 tokens, [slot][256]; a tile of TM < 256
  // rows starts inside such a block; waves past the tile's rows repeat the
  // loads of the waves before them into the same LDS words, so every wave
  // issues the same number of loads per stage)
  const bool arat = NW == 4 || wid < 4;
  const int bw = (NW == 8 ? wid - 4 : wid) % (TM / 64);
  const int64_t gb_off = (m0 / kTM) * a.nslot * kTM + m0 % kTM;
  const __amdgpu_buffer_rsrc_t rrat = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(a.ratio + vt * a.nslot * kTN), 0, a.nslot * kTN * 4, kBufferWord3);
  const __amdgpu_buffer_rsrc_t rbias = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(a.gbias + gb_off), 0, int(a.nslot * kTM - m0 % kTM) * 4, kBufferWord3);

  // per-lane load offsets (row and swizzled 16-byte unit) of the residual
  // stages; the expansion stages use the same units with their own row
  // strides; the stage's k offset is added per stage
  auto xunit = [&](int i, uint32_t stride) {
    const int off = (wid * G::NX + i) * 1024 + 16 * lane;
    const int r = off / (2 * kKS), p = (off % (2 * kKS)) / 16;
    return uint32_t(r < rows ? r : rows - 1) * stride + 16u * uint32_t(p ^ swz_x(r));
  };
  auto cunit = [&](int ci, uint32_t stride) {
    const int off = (wid * G::NC + ci) * 1024 + 16 * lane;
    const int c = off / (kKS / 2), p = (off % (kKS / 2)) / 16;
    return uint32_t(c < cols ? c : cols - 1) * stride + 16u * uint32_t(p ^ swz_c(c));
  };
  uint32_t xo[G::NX];
#pragma unroll
  for (int i = 0; i < G::NX; ++i) xo[i] = xunit(i, ldx2);
  uint32_t co[G::NC];
#pragma unroll
  for (int ci = 0; ci < G::NC; ++ci) co[ci] = cunit(ci, rowbytes);
  // dense-row units, laid out like x (rows of kKS bf16, XOR-swizzled units)
  auto dunit = [&](int i) {
    const int off = (wid * G::ND + i) * 1024 + 16 * lane;
    const int r = off / (2 * kKS), p = (off % (2 * kKS)) / 16;
    return uint32_t(r < cols ? r : cols - 1) * dstride + 16u * uint32_t(p ^ swz_x(r));
  };
  uint32_t dof[G::ND > 0 ? G::ND : 1];
#pragma unroll
  for (int i = 0; i < G::ND; ++i) dof[i] = dunit(i);
  const uint32_t ao_rat = uint32_t((wid & 3) * 64 + lane) * 4;
  const uint32_t ao_bias = uint32_t(bw * 64 + lane < rows ? bw * 64 + lane : rows - 1) * 4;

  const int nst = a.d / kKS, spg = a.g / kKS, ntot = nst + a.nch;
  const int slot_u = ngrp, slot_a = ngrp + (a.nch_u > 0 ? 1 : 0);
  auto slot_of = [&](int s) {
    return s < nst ? s / spg : (s - nst < a.nch_u ? slot_u : slot_a);
  };
  // load PART (0 .. NL-1) of this wave's share of stage s into ring slot
  // buf: x (or t) units, code units, then the ratio / bias units.  KIND: 1
  // a residual stage, 2 an expansion stage, 3 either (checked).
  auto issue_part = [&](int s, int buf, int part, auto kind) {
    constexpr int KIND = decltype(kind)::value;
    lds_u8* base = L + buf * G::STAGE;
    const bool res = KIND == 1 || (KIND == 3 && s < nst);
    if (part < G::NX) {
      lds_u8* dst = base + (wid * G::NX + part) * 1024;
      if (res) dma16(rx, dst, xo[part] + uint32_t(s) * (kKS * 2));
      else dma16(rt, dst, xunit(part, trow) + uint32_t(s - nst) * 128);
    } else if (part < G::NX + G::NC) {
      const int ci = part - G::NX;
      lds_u8* dst = base + G::XBYTES + (wid * G::NC + ci) * 1024;
      if (res) dma16(rc, dst, co[ci] + uint32_t(s) * (kKS / 2));
      else dma16(ru, dst, cunit(ci, urow) + uint32_t(s - nst) * 32);
    } else if (part < G::NX + G::NC + G::NA) {
      const uint32_t k = uint32_t(KIND == 1 ? s / spg : slot_of(s)) * 1024u;
      if (NW == 4 ? part == G::NX + G::NC : arat)
        dma4(rrat, base + G::RAT + (wid & 3) * 256, ao_rat + k);
      else
        dma4(rbias, base + G::BIAS + bw * 256, ao_bias + k);
    } else {
      const int di = part - G::NX - G::NC - G::NA;
      lds_u8* dst = base + G::DOFF + (wid * G::ND + di) * 1024;
      if (res) dma16(rd, dst, dof[di] + uint32_t(s) * (kKS * 2));
      else dma16(rdz, dst, 0u);
    }
  };
  using kMain = std::integral_constant<int, 1>;
  using kExp = std::integral_constant<int, 2>;
  using kAny = std::integral_constant<int, 3>;
  using kNone = std::integral_constant<int, 0>;
  auto issue = [&](int s, int buf) {
#pragma unroll
    for (int part = 0; part < G::NL; ++part) issue_part(s, buf, part, kAny{});
  };

  // fragment offsets within a stage: residual stages take x chunks 2q + kc,
  // expansion stages chunk 4 kc + q ([hi | mid] for kc = 0, [lo | 0] for
  // kc = 1), matched by code dimensions 8 (q % 2) .. +7 of [c | c]
  const uint32_t arow = uint32_t(WM * wm + lr) * (2 * kKS);
  uint32_t aoff[2];
#pragma unroll
  for (int kc = 0; kc < 2; ++kc) aoff[kc] = arow + 16u * uint32_t((2 * q + kc) ^ swz_x(lr));
  const uint32_t boff =
      G::XBYTES + uint32_t(64 * wn + lr) * 32 + 16u * uint32_t((q >> 1) ^ swz_c(lr)) + 8u * (q & 1);

  f32x4_t acc[MI][4];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // the dense head's logits (fidelity pass): plain fp32 sums of bf16 products
  constexpr int MD = XE == 1 ? MI : 1;
  f32x4_t accd[MD][4];
#pragma unroll
  for (int i = 0; i < MD; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) accd[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // dense B fragments: row 64 wn + 16 ni + lr, the same 16-byte units as x
  uint32_t bdoff[2];
#pragma unroll
  for (int kc = 0; kc < 2; ++kc)
    bdoff[kc] = G::DOFF + uint32_t(64 * wn + lr) * (2 * kKS) + 16u * uint32_t((2 * q + kc) ^ swz_x(lr));

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
  // MFMAs of stage s (one per row block of its first K-chunk, then of the
  // second where a wave has more loads than row blocks), so the waves'
  // vector-memory traffic does not queue up in one burst after the barrier.
  int buf = 0;   // ring slot of the next stage to compute
  auto next_stage = [&](int s) {
    if (s + 1 < ntot) wait_loads_barrier<G::NL>();
    else wait_loads_barrier<0>();
    const lds_u8* base = L + buf * G::STAGE;
    buf = buf == 2 ? 0 : buf + 1;
    return base;
  };

  // slot start: rescale to the slot's scale and add its bias
  auto rescale = [&](const lds_u8* base) {
    float rat[4];
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) rat[ni] = lds_load<float>(base + G::RAT + (64 * wn + 16 * ni + lr) * 4);
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
      const f32x4_t bias = lds_load<f32x4_t>(base + G::BIAS + (WM * wm + 16 * mi + 4 * q) * 4);
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
    bf16x8_t A[MI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) A[mi] = lds_load<bf16x8_t>(base + aoff[0] + mi * 32 * kKS);
    if (sg == 0) rescale(base);
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      bf16x8_t B[4];
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) B[ni] = unpack8(braw[ni][kc], kMask, kMagic);
      bf16x8_t Bd[XE == 1 ? 4 : 1];
      if constexpr (XE == 1) {
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          Bd[ni] = lds_load<bf16x8_t>(base + bdoff[kc] + ni * 16 * (2 * kKS));
      }
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) {
        const bf16x8_t Am = A[mi];
        if (kc == 0) A[mi] = lds_load<bf16x8_t>(base + aoff[1] + mi * 32 * kKS);
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Am, B[ni], acc[mi][ni], 0, 0, 0);
        if constexpr (XE == 1) {
#pragma unroll
          for (int ni = 0; ni < 4; ++ni)
            accd[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Am, Bd[ni], accd[mi][ni], 0, 0, 0);
        }
#pragma unroll
        for (int pp = 0; pp < G::PPS; ++pp) {
          const int part = (kc * MI + mi) * G::PPS + pp;
          if (part < G::NL) {
            if constexpr (ISSUE == 1) issue_part(s + 2, nb, part, kMain{});
            if constexpr (ISSUE == 3) if (s + 2 < ntot) issue_part(s + 2, nb, part, kAny{});
          }
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
      for (int mi = 0; mi < MI; ++mi) {
        const bf16x8_t A = lds_load<bf16x8_t>(base + eoff + mi * 32 * kKS);
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B[ni], acc[mi][ni], 0, 0, 0);
#pragma unroll
        for (int pp = 0; pp < G::PPS; ++pp) {
          const int part = (kc * MI + mi) * G::PPS + pp;
          if (part < G::NL) {
            if constexpr (ISSUE == 2) issue_part(s + 2, nb, part, kExp{});
            if constexpr (ISSUE == 3) if (s + 2 < ntot) issue_part(s + 2, nb, part, kAny{});
          }
        }
      }
    }
  };
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
    for (int mi = 0; mi < MI; ++mi) acc[mi][ni] *= fin[ni];

  // ---- epilogue
  if constexpr (XE == 1) {
    // per token row of the tile: the FidTilePart of its valid columns (a the
    // dense logit, b the packed one); the 16 lanes of a quarter-wave share
    // rows, the four waves along the vocabulary merge through LDS in order
    FidTilePart* sp = reinterpret_cast<FidTilePart*>(mfma_lds);   // [4][TM]
    __syncthreads();
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = WM * wm + 16 * mi + 4 * q + i;
        float ma = -INFINITY, mb = -INFINITY;
        int ia = kNoIdx;
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          const int col = 64 * wn + 16 * ni + lr;
          if (col < cols) {
            const float av = accd[mi][ni][i];
            if (av > ma) {   // strict: a lane's columns rise, so its first maximum stays
              ma = av;
              ia = col;
            }
            mb = fmaxf(mb, acc[mi][ni][i]);
          }
        }
        const float mar = row16_max(ma);
        const int iar = row16_min_i(ma == mar ? ia : kNoIdx);
        const float mbr = row16_max(mb);
        float bat = -INFINITY, sa = 0.f, sb = 0.f, t = 0.f, sq = 0.f;
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          const int col = 64 * wn + 16 * ni + lr;
          if (col < cols) {
            const float av = accd[mi][ni][i], bv = acc[mi][ni][i];
            if (col == iar) bat = bv;
            const float ea = expf(av - mar), dd = av - bv;
            sa += ea;
            sb += expf(bv - mbr);
            t += ea * dd;
            sq += dd * dd;
          }
        }
        bat = row16_max(bat);
        sa = row16_sum(sa);
        sb = row16_sum(sb);
        t = row16_sum(t);
        sq = row16_sum(sq);
        if (lr == 0) sp[wn * TM + row] = FidTilePart{mar, mbr, bat, sa, sb, t, sq, iar};
      }
    __syncthreads();
    if (tid < rows) {
      FidTilePart r = sp[tid];   // wave 0 holds column 0, always valid
#pragma unroll
      for (int w = 1; w < 4; ++w) {
        const FidTilePart o = sp[w * TM + tid];
        if (o.ma > r.ma) {
          const float f = expf(r.ma - o.ma);
          r.sa = r.sa * f + o.sa;
          r.t = r.t * f + o.t;
          r.ma = o.ma;
          r.ia = o.ia;
          r.bat = o.bat;
        } else if (o.ma > -INFINITY) {   // equal maxima keep the smaller index (this wave's)
          const float f = expf(o.ma - r.ma);
          r.sa += o.sa * f;
          r.t += o.t * f;
        }
        if (o.mb > r.mb) {
          r.sb = r.sb * expf(r.mb - o.mb) + o.sb;
          r.mb = o.mb;
        } else if (o.mb > -INFINITY) {
          r.sb += o.sb * expf(o.mb - r.mb);
        }
        r.sq += o.sq;
      }
      r.ia = r.ia == kNoIdx ? kNoIdx : int(v0) + r.ia;
      reinterpret_cast<FidTilePart*>(a.fid_part)[(m0 + tid) * a.n_vt + vt] = r;
    }
  } else if constexpr (XE == 2) {
    // per token row: the packed logits of this tile ranked ahead of the
    // reference's top-1 (larger, or equal at a smaller index), added to rank
    float* sbr = reinterpret_cast<float*>(mfma_lds);   // [TM] bref
    int* sri = reinterpret_cast<int*>(sbr + TM);       // [TM] ref_idx - v0, clamped
    int* scnt = sri + TM;                              // [4][TM]
    __syncthreads();
    if (tid < TM) {
      const bool ok = tid < rows;
      const int64_t dr = ok ? a.ref_idx[m0 + tid] - v0 : -1;
      sbr[tid] = ok ? a.bref[m0 + tid] : 0.f;
      sri[tid] = dr < 0 ? -1 : (dr > kTN ? kTN : int(dr));
    }
    __syncthreads();
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = WM * wm + 16 * mi + 4 * q + i;
        const float br = sbr[row];
        const int ri = sri[row];
        int c = 0;
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          const int col = 64 * wn + 16 * ni + lr;
          const float bv = acc[mi][ni][i];
          c += (col < cols) & ((bv > br) | ((bv == br) & (col < ri)));
        }
#pragma unroll
        for (int off = 8; off > 0; off >>= 1) c += __shfl_xor(c, off, 16);
        if (lr == 0) scnt[wn * TM + row] = c;
      }
    __syncthreads();
    if (tid < rows) {
      const int tot = scnt[tid] + scnt[TM + tid] + scnt[2 * TM + tid] + scnt[3 * TM + tid];
      if (tot) atomicAdd(reinterpret_cast<unsigned long long*>(a.rank + m0 + tid),
                         (unsigned long long)tot);
    }
  } else if constexpr (!CE) {
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = WM * wm + 16 * mi + 4 * q + i;
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
    float2* sred = reinterpret_cast<float2*>(mfma_lds);               // [4][TM]
    int* sy = reinterpret_cast<int*>(mfma_lds + 4 * TM * sizeof(float2));    // [TM]
    int* sidx = sy + TM;                                                 // [4][TM] argmax
    __syncthreads();
    if (tid < TM) sy[tid] = y_row >= v0 && y_row < v0 + cols ? int(y_row - v0) : -1;
    __syncthreads();
    // IDX: also the smallest tile column at each row's maximum (argmax
    // partials); compiled apart so the CE-only pass pays nothing for it
    auto rows_pass = [&](auto IDX) {
      constexpr bool kIdx = decltype(IDX)::value;
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = WM * wm + 16 * mi + 4 * q + i;
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
            sred[wn * TM + row] = make_float2(mx, se);
            if constexpr (kIdx) sidx[wn * TM + row] = ai;
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
      for (int w = 1; w < 4; ++w) lse_merge(m_, s_, sred[w * TM + tid].x, sred[w * TM + tid].y);
      a.part[(m0 + tid) * a.n_vt + vt] = make_float2(m_, s_);
      if (a.part_idx) {
        int ai = kNoIdx;
#pragma unroll
        for (int w = 0; w < 4; ++w)
          if (sred[w * TM + tid].x == m_) ai = min(ai, sidx[w * TM + tid]);
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
  int cu_row;            // bytes per row of U_c (r_c int8 codes, or ARCHEAD_I5 words)
  int u5;                // U_c codes are ARCHEAD_I5 words
};

__device__ __forceinline__ float nz_scale(uint16_t h) {
  const float s = f16_to_f32(h);
  return s == 0.f ? kZeroScale : s;
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

}  // namespace
