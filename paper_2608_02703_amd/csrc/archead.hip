// ARCHead packed LM-head forward on gfx950: the C ABI's compute entry points
// (argument checks, workspace layout, kernel choice and launches; the kernel
// templates are in dev_*.cuh, instantiated in k_*.hip).
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
#include "kernels.h"
#include "dev_gemv.cuh"
#include "dev_dec.cuh"
#include "dev_mid.cuh"
#include "dev_mfma.cuh"

namespace {

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

// ------------------------------------------------------------ dispatch
size_t gemv_lds_bytes(const archead_desc& d, int tok) {
  // x, the chunk biases, and one copy of t per wave (U_c and A_w parts each
  // padded to a multiple of 4 dimensions)
  const size_t rp = size_t(4 * ((d.r_c + 3) / 4 + (d.r_r + 3) / 4));
  return size_t(tok) * (size_t(d.d) * 2 + size_t(d.d / 32) * 4 + size_t(kWaves) * rp * 4);
}

bool aligned(const void* p, size_t a);

// Whether the GEMV's pipelined path applies to the head (expansion codes of
// a row fit the segment as dwords, d/g groups fit a step's scale load), and
// whether it runs the variant for general factor codes (a rank that is not
// a multiple of 4, or ARCHEAD_I5 core-left codes; built for 8 and 16 lanes
// per row).  Heads it does not apply to take the byte-wise path throughout.
struct GemvMode {
  bool fast = false;
  int gen = 0;   // kern::gemv's factor-code variant
};
GemvMode gemv_mode(const archead_handle* h) {
  const archead_desc& d = h->desc;
  const int lpr = archead::lanes_per_row(d);
  const int kd = lpr >= 64 ? 1 : 2;   // ExpLanes<LPR>::KD
  const int64_t ngrp = d.d / d.g;
  const bool sc8 = d.scale_dtype == ARCHEAD_U8;
  const int64_t gpl = sc8 ? 4 : 2;    // a step's scales: groups per segment lane
  const int64_t rq = (d.r_c + 3) / 4 + (d.r_r + 3) / 4;
  GemvMode m;
  const bool shape = rq <= int64_t(kd) * lpr && ngrp % gpl == 0 && ngrp <= gpl * lpr;
  if (archead::gen_codes(d)) {
    // the general reads take 32-bit offsets into the factor-code buffers
    const bool fits = d.V * (archead::core_u_row_bytes(d) + 8) < (int64_t(1) << 31) &&
                      d.V * (d.r_r + 8) < (int64_t(1) << 31);
    m.fast = shape && fits && (lpr == 8 || lpr == 16);
    m.gen = m.fast ? archead::gen_codes(d) : 0;
  } else {
    m.fast = shape && (d.r_c == 0 || aligned(h->ptrs.core_u, 4)) &&
             (d.r_r == 0 || aligned(h->ptrs.corr_a, 4));
  }
  return m;
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

int64_t gemv_grid(const archead_handle* h, int tok, bool ce, bool topk) {
  const bool sc8 = h->desc.scale_dtype == ARCHEAD_U8;
  const int gen = gemv_mode(h).gen;
  const int slot = (topk ? 64 : 0) + (gen ? 32 : 0) + (sc8 ? 16 : 0) + (ce ? 8 : 0) + tok;
  archead_handle* mh = const_cast<archead_handle*>(h);
  int cached = mh->grid_cache[slot].load(std::memory_order_relaxed);
  const int64_t steps = (h->desc.V + gemv_rows_per_step(h->desc) - 1) / gemv_rows_per_step(h->desc);
  const int64_t max_blocks = (steps + kWaves - 1) / kWaves;
  if (cached <= 0) {
    const int lpr = lanes_per_row(h->desc);
    const void* fn = topk ? kern::gemv_topk(lpr, sc8, gen) : kern::gemv(tok, lpr, ce, sc8, gen);
    int nb = 0;
    const size_t lds = gemv_lds_bytes(h->desc, tok);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fn,
                                                     kBlock, lds) != hipSuccess ||
        nb <= 0)
      nb = 1;
    // a few resident workgroups per CU stream best (a launch setting may
    // choose another count)
    const int64_t bpc = h->launch[ARCHEAD_LAUNCH_GEMV_BLOCKS_PER_CU].load(std::memory_order_relaxed);
    const int want = bpc > 0 ? int(bpc) : kGemvBlocksPerCu;
    if (nb > want) nb = want;
    // every resident wave (measured faster than fewer waves with an even
    // split of the steps)
    cached = nb * h->n_cu;
    const int64_t grid = h->launch[ARCHEAD_LAUNCH_GEMV_GRID].load(std::memory_order_relaxed);
    if (grid > 0) cached = int(grid);
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
  if (const int64_t c = h->launch[ARCHEAD_LAUNCH_DEC_BLOCKS].load(std::memory_order_relaxed)) cap = c;
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
  if (const int64_t c = h->launch[ARCHEAD_LAUNCH_MID_BLOCKS].load(std::memory_order_relaxed)) cap = c;
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

// Whether a top-k call of M tokens runs fused in the single-token GEMV.
// The merge of per-partial top-k lists: k rounds of a workgroup-wide best
// when every thread holds at most kTopKMergeC candidates, else the scan
// (floor, per-wave lists, wave-ordered merge).
static hipError_t launch_topk_merge(int64_t n_part, int k, int64_t rows, void** args,
                                    hipStream_t s) {
  // four waves while they hold every candidate (a round's barrier and
  // cross-wave step are cheaper), else sixteen
  if (n_part * k <= int64_t(256) * kTopKMergeC)
    return hipLaunchKernel(kern::topk_merge(256), dim3(unsigned(rows)), dim3(256), args, 0, s);
  if (n_part * k <= int64_t(kTopKMergeBlock) * kTopKMergeC)
    return hipLaunchKernel(kern::topk_merge(kTopKMergeBlock), dim3(unsigned(rows)),
                           dim3(kTopKMergeBlock), args, 0, s);
  return hipLaunchKernel(kern::topk_merge_scan(), dim3(unsigned(rows)), dim3(kBlock), args, 0, s);
}

bool topk_fused(const archead_handle* h, int64_t M) {
  return M == 1 && choose_path(h, 1) == Path::kGemv &&
         kern::gemv_topk(lanes_per_row(h->desc), h->desc.scale_dtype == ARCHEAD_U8,
                         gemv_mode(h).gen) != nullptr;
}

// Slices per token row of the top-k of a chunk of logits: enough that the
// chunk's rows give about a thousand workgroups, at most 64.
int64_t topk_row_parts(int64_t chunk) {
  const int64_t np = (1024 + chunk - 1) / chunk;
  return np < 1 ? 1 : (np > 64 ? 64 : np);
}

static WsLayout topk_layout(const archead_handle* h, int64_t M) {
  WsLayout w;
  const archead_desc& d = h->desc;
  size_t off = 0;
  int64_t rows = 1;
  if (topk_fused(h, M)) {
    w = ws_layout(h, 1, ARCHEAD_OP_LOGITS);   // the GEMV's stage-1 words
    off = w.total;
    w.tk_fused = true;
    w.n_part = gemv_grid(h, 1, false, true);
  } else {
    const int64_t chunk = M < kTopKChunk ? M : kTopKChunk;
    w.tk_chunk = chunk;
    w.tk_lg_off = 0;
    off = align256(sizeof(float) * size_t(chunk) * size_t(d.V));
    w.tk_in_off = off;
    // every chunk runs on the kernel the whole call would take, so the
    // logits are those archead_logits gives for the same M
    w.tk_path = choose_path(h, M);
    size_t inner = ws_layout_path(h, chunk, ARCHEAD_OP_LOGITS, w.tk_path).total;
    if (M % chunk) {
      const size_t t = ws_layout_path(h, M % chunk, ARCHEAD_OP_LOGITS, w.tk_path).total;
      inner = t > inner ? t : inner;
    }
    off = align256(off + inner);
    w.n_part = topk_row_parts(chunk);
    rows = chunk;
  }
  const size_t lists = size_t(rows) * size_t(w.n_part) * kTopKMaxK;
  w.tk_pv_off = off;
  off = align256(off + sizeof(float) * lists);
  w.tk_pi_off = off;
  off = align256(off + sizeof(int32_t) * lists);
  w.total = off;
  return w;
}

WsLayout ws_layout(const archead_handle* h, int64_t M, archead_op op) {
  if (h && M > 0 && op == ARCHEAD_OP_TOPK) return topk_layout(h, M);
  if (h && M > 0 && op == ARCHEAD_OP_FIDELITY) {
    WsLayout w = ws_layout_path(h, M, ARCHEAD_OP_LOGITS, Path::kTiled);
    const size_t n_vt = size_t((h->desc.V + kTN - 1) / kTN);
    w.fid_off = w.total;
    w.bref_off = align256(w.fid_off + 32 * size_t(M) * n_vt);
    w.total = align256(w.bref_off + sizeof(float) * size_t(M));
    return w;
  }
  return ws_layout_path(h, M, op, h ? choose_path(h, M) : Path::kGemv);
}

// The layout for M tokens on the kernel `path`.
WsLayout ws_layout_path(const archead_handle* h, int64_t M, archead_op op, Path path) {
  WsLayout w;
  if (!h || M <= 0) return w;
  const archead_desc& d = h->desc;
  size_t off = 0;
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
  p.cu_row = int(core_u_row_bytes(d));
  p.u5 = d.core_u_dtype == ARCHEAD_I5;
  p.ucodes = reinterpret_cast<int8_t*>(base + pl.uc_off);
  const int64_t work = std::max({p.n_vt * kTN, int64_t(R) * d.d / 8, d.V * (p.urow / 16)});
  const int64_t pblocks =
      std::max<int64_t>(1, std::min<int64_t>((work + kBlock - 1) / kBlock, 4 * int64_t(h->n_cu)));
  void* args[] = {&p};
  hipError_t e = hipLaunchKernel(kern::prep(), dim3(unsigned(pblocks)), dim3(kBlock), args, 0, s);
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
  void* args[] = {&a};
  hipError_t e = hipLaunchKernel(kern::stage1m(),
                                 dim3(unsigned(mblocks), unsigned(rblocks), unsigned(a.ksplit)),
                                 dim3(kS1MBlock), args, 0, s);
  if (e == hipSuccess && a.ksplit > 1) {
    const int64_t n = M * R;
    e = hipLaunchKernel(kern::stage1m_fin(), dim3(unsigned((n + kBlock - 1) / kBlock)),
                        dim3(kBlock), args, 0, s);
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
  {
    const int64_t sl = h->launch[ARCHEAD_LAUNCH_T_SPIN_LIMIT].load(std::memory_order_relaxed);
    o.spin_limit = sl >= 0 ? int(sl) : kDefaultSpinLimit;
  }
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
  const bool sc8 = d.scale_dtype == ARCHEAD_U8;
  a.fast = gemv_mode(h).fast;
  a.u5 = d.core_u_dtype == ARCHEAD_I5;
  a.rrs = sc8 ? static_cast<const uint16_t*>(h->ptrs.res_row_scales) : a.rs;
  // an absent factor reads the (valid, 16-byte aligned) residual buffers with
  // stride 0 instead; its contribution is masked to zero in the kernel
  a.cu_stride = core_u_row_bytes(d); a.su_stride = d.r_c ? 1 : 0;
  a.cu_bytes = d.V * a.cu_stride;
  a.ca_bytes = d.V * d.r_r;
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
                                  int64_t forced_grid, hipStream_t s, bool topk = false) {
  const int lpr = lanes_per_row(h->desc);
  // timing events (if set) are attached to the first and last dispatch
  // packets themselves, so they bracket exactly the kernel execution
  hipEvent_t ev0 = static_cast<hipEvent_t>(h->ev_start.load(std::memory_order_relaxed));
  hipEvent_t ev1 = static_cast<hipEvent_t>(h->ev_stop.load(std::memory_order_relaxed));
  for (int64_t m0 = 0; m0 < M; m0 += 4) {
    const int tok = int(M - m0 < 4 ? M - m0 : 4);
    const bool sc8 = h->desc.scale_dtype == ARCHEAD_U8;
    const void* fn = topk ? kern::gemv_topk(lpr, sc8, gemv_mode(h).gen)
                          : kern::gemv(tok, lpr, ce, sc8, gemv_mode(h).gen);
    const int64_t grid = a.n_prod_blocks + (forced_grid > 0 ? forced_grid : gemv_grid(h, tok, ce));
    a.tok0 = m0;
    const size_t lds = gemv_lds_bytes(h->desc, tok);
    if (lds > 65536) {
      hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
      if (e != hipSuccess) return hip_fail(e, "LDS size attribute");
    }
    void* args[] = {&a};
    const bool first = m0 == 0, last = m0 + 4 >= M;
    hipError_t e = hipExtLaunchKernel(fn, dim3(unsigned(grid)),
                                      dim3(kBlock), args, lds, s, first ? ev0 : nullptr,
                                      last ? ev1 : nullptr, 0);
    if (e != hipSuccess) return hip_fail(e, "GEMV launch");
  }
  return ARCHEAD_OK;
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
  const void* fn = kern::dec(gw, ce, l0.kcu <= 2 && l0.kca <= 2 ? 2 : 4, sc8, gen_codes(d));
  a.cu_row = int(core_u_row_bytes(d));
  a.u5 = d.core_u_dtype == ARCHEAD_I5;
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
      hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, l.total);
      if (e != hipSuccess) return hip_fail(e, "decode LDS size attribute");
    }
    void* args[] = {&a};
    const bool first = m0 == 0, last = m0 + tpp >= M;
    hipError_t e = hipExtLaunchKernel(fn, dim3(unsigned(grid)),
                                      dim3(kDBlock), args, size_t(l.total), s,
                                      first ? ev0 : nullptr, last ? ev1 : nullptr, 0);
    if (e != hipSuccess) return hip_fail(e, "MFMA decode launch");
  }
  return ARCHEAD_OK;
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
  a.cu_row = int(core_u_row_bytes(d));
  a.u5 = d.core_u_dtype == ARCHEAD_I5;
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
    const void* fn = kern::mid(gw, ce, sc8, gen_codes(d));
    const MidLds l = mid_lds(d);
    a.tok0 = m0;
    a.M = tok;
    a.kcu = l.kcu; a.kca = l.kca;
    a.tstr = l.tstr;
    a.off_bias = l.off_bias; a.off_red = l.off_red; a.off_y = l.off_y; a.off_idx = l.off_idx;
    a.off_sc = l.off_sc;
    if (l.total > 65536) {
      hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, l.total);
      if (e != hipSuccess) return hip_fail(e, "several-token LDS size attribute");
    }
    void* args[] = {&a};
    const bool first = m0 == 0, last = m0 + kMidTokMax >= M;
    hipError_t e = hipExtLaunchKernel(fn, dim3(unsigned(grid)),
                                      dim3(kMidBlock), args, size_t(l.total), s,
                                      first ? ev0 : nullptr, last ? ev1 : nullptr, 0);
    if (e != hipSuccess) return hip_fail(e, "several-token launch");
  }
  return ARCHEAD_OK;
}

// Token rows per tile of the 8-wave tiled kernel: 128 for calls of at most
// 128 tokens (the 256-row tile would spend half or more of its MFMA work on
// padding rows), else 256.
int tiled_tm(int64_t M) { return M <= 128 ? 128 : kTM; }

// Tile rows and waves per workgroup of the tiled kernel for a call of M
// tokens: 64-row tiles of 4 waves, three workgroups per CU, up to
// kTiled64MaxM tokens; 128-row tiles of 4 waves, two workgroups per CU, up
// to kTiledNw4MaxM tokens (measured 10-25% faster than one workgroup of 8
// waves per CU at M = 16 .. 1024, where tile starts, LDS waits and the
// epilogue would leave the matrix unit idle); above, 256-row tiles of 8
// waves (equal at M = 4096, where the chip runs at its power limit).
// The launch settings ARCHEAD_LAUNCH_TILE_WAVES (4 or 8) and
// ARCHEAD_LAUNCH_TILE_ROWS (64 or 128, with 4 waves) override the choice.
constexpr int64_t kTiled64MaxM = 64;
constexpr int64_t kTiledNw4MaxM = 1024;
struct TiledShape { int tm, nw; };
TiledShape tiled_shape(const archead_handle* h, int64_t M) {
  TiledShape t = M <= kTiled64MaxM    ? TiledShape{64, 4}
                 : M <= kTiledNw4MaxM ? TiledShape{128, 4}
                                      : TiledShape{kTM, 8};
  const int64_t nw = h->launch[ARCHEAD_LAUNCH_TILE_WAVES].load(std::memory_order_relaxed);
  const int64_t tm = h->launch[ARCHEAD_LAUNCH_TILE_ROWS].load(std::memory_order_relaxed);
  if (nw == 4) t = TiledShape{128, 4};
  else if (nw == 8) t = TiledShape{tiled_tm(M), 8};
  if (t.nw == 4 && (tm == 64 || tm == 128)) t.tm = int(tm);
  return t;
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
  const int tm = tiled_shape(h, M).tm;
  a.n_mt = (M + tm - 1) / tm;
  a.n_vt = (d.V + kTN - 1) / kTN;
  a.n_tiles = a.n_vt * a.n_mt;
  a.tiles_per_xcd = (a.n_tiles + 7) / 8;
  return a;
}

archead_status launch_mfma(const archead_handle* h, MfmaArgs& a, bool ce, hipStream_t s) {
  // byte ranges of one tile's buffers must stay below 2 GiB
  if (int64_t(kTM) * a.ldx * 2 >= (int64_t(1) << 31))
    return fail(ARCHEAD_E_UNSUPPORTED, "ldx too large for the many-token kernel");
  const TiledShape ts = tiled_shape(h, a.M);
  const void* fn = kern::mfma(ce, ts.tm, ts.nw);
  const int lds = ts.nw == 4 ? (ts.tm == 64 ? MGeomT<64, 4>::LDS : MGeomT<128, 4>::LDS)
                  : ts.tm == 128 ? MGeomT<128>::LDS : MGeom::LDS;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return hip_fail(e, "MFMA LDS size attribute");
  hipEvent_t ev0 = static_cast<hipEvent_t>(h->ev_start.load(std::memory_order_relaxed));
  hipEvent_t ev1 = static_cast<hipEvent_t>(h->ev_stop.load(std::memory_order_relaxed));
  void* args[] = {&a};
  const int64_t grid = 8 * a.tiles_per_xcd;
  if (grid > 0x7fffffff) return fail(ARCHEAD_E_UNSUPPORTED, "too many MFMA tiles");
  e = hipExtLaunchKernel(fn, dim3(unsigned(grid)), dim3(unsigned(ts.nw * 64)), args, size_t(lds), s,
                         ev0, ev1, 0);
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

// The logits of archead_logits after its checks (also the first half of
// the unfused top-k).
archead_status logits_run(const archead_handle* h, const void* x, int64_t M, int64_t ldx,
                          void* out, archead_dtype out_dtype, int64_t ldo, void* ws,
                          hipStream_t s, Path path) {
  archead_status st = ARCHEAD_OK;
  const WsLayout w = ws_layout_path(h, M, ARCHEAD_OP_LOGITS, path);
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
  if (d.r_c && d.core_u_dtype == ARCHEAD_I5 && !aligned(ptrs->core_u, 4))
    return fail(ARCHEAD_E_MISALIGNED, "ARCHEAD_I5 core_u must be 4-byte aligned");
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
  for (auto& k : h->launch) k.store(0);
  h->launch[ARCHEAD_LAUNCH_T_SPIN_LIMIT].store(-1);
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
  return logits_run(h, x, M, ldx, out, out_dtype, ldo, ws, static_cast<hipStream_t>(stream),
                    choose_path(h, M));
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

archead_status archead_logit_fidelity_head(const archead_handle* h, const void* x, int64_t M,
                                           int64_t ldx, const void* dense, int64_t ldw,
                                           float* kl, float* sq, int64_t* ref_idx,
                                           int64_t* rank, void* ws, size_t ws_bytes,
                                           void* stream) {
  clear_error();
  archead_status st = check_call(h, x, M, ldx, ws, ws_bytes, ARCHEAD_OP_FIDELITY);
  if (st != ARCHEAD_OK || M == 0) return st;
  if (!mfma_ok(h)) return fail(ARCHEAD_E_UNSUPPORTED, "the head has no tiled kernel (g %% 64 != 0)");
  if (!dense || !kl || !sq || !ref_idx || !rank)
    return fail(ARCHEAD_E_INVALID_ARG, "dense, kl, sq, ref_idx and rank are required");
  if (ldw < h->desc.d) return fail(ARCHEAD_E_INVALID_ARG, "ldw < d");
  if (!aligned(dense, 16) || ldw % 8)
    return fail(ARCHEAD_E_MISALIGNED, "dense must be 16-byte aligned with ldw %% 8 == 0");
  if (!aligned(kl, 4) || !aligned(sq, 4) || !aligned(ref_idx, 8) || !aligned(rank, 8))
    return fail(ARCHEAD_E_MISALIGNED, "kl / sq / ref_idx / rank misaligned");
  if (ldw * 2 * kTN >= (int64_t(1) << 31))
    return fail(ARCHEAD_E_UNSUPPORTED, "ldw too large for the tiled kernel");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const WsLayout w = ws_layout(h, M, ARCHEAD_OP_FIDELITY);
  char* base = static_cast<char*>(ws);
  st = launch_mfma_prologue(h, x, M, ldx, w, base, s);
  if (st != ARCHEAD_OK) return st;
  MfmaArgs a = mfma_args(h, x, M, ldx, w, base);
  a.n_mt = (M + 63) / 64;   // 64-row tiles of 4 waves in both passes
  a.n_tiles = a.n_vt * a.n_mt;
  a.tiles_per_xcd = (a.n_tiles + 7) / 8;
  a.dense = static_cast<const uint16_t*>(dense);
  a.ldw = ldw;
  a.fid_part = base + w.fid_off;
  float* bref = reinterpret_cast<float*>(base + w.bref_off);
  a.bref = bref;
  a.ref_idx = ref_idx;
  a.rank = rank;
  const int64_t grid = 8 * a.tiles_per_xcd;
  if (grid > 0x7fffffff) return fail(ARCHEAD_E_UNSUPPORTED, "too many MFMA tiles");
  for (int xe = 1; xe <= 2; ++xe) {
    const void* fn = kern::mfma_fid(xe);
    const int lds = xe == 1 ? MGeomT<64, 4, true>::LDS : MGeomT<64, 4>::LDS;
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return hip_fail(e, "fidelity pass LDS size attribute");
    void* args[] = {&a};
    e = hipExtLaunchKernel(fn, dim3(unsigned(grid)), dim3(256), args, size_t(lds), s, nullptr,
                           nullptr, 0);
    if (e != hipSuccess) return hip_fail(e, "fidelity pass launch");
    if (xe == 1) {
      const FidTilePart* part = static_cast<const FidTilePart*>(a.fid_part);
      int64_t n_vt = a.n_vt;
      void* margs[] = {&part, &n_vt, &M, &kl, &sq, &ref_idx, &bref, &rank};
      e = hipLaunchKernel(kern::fid_head_merge(), dim3(unsigned((M + 63) / 64)), dim3(64), margs,
                          0, s);
      if (e != hipSuccess) return hip_fail(e, "fidelity merge launch");
    }
  }
  return ARCHEAD_OK;
}

archead_status archead_logits_topk(const archead_handle* h, const void* x, int64_t M,
                                   int64_t ldx, int32_t k, float* vals, int64_t* idx,
                                   int64_t ldk, void* ws, size_t ws_bytes, void* stream) {
  clear_error();
  if (h && (k < 1 || k > kTopKMaxK || int64_t(k) > h->desc.V))
    return fail(ARCHEAD_E_INVALID_ARG, "k = %d is outside 1 .. min(%d, V)", int(k), kTopKMaxK);
  archead_status st = check_call(h, x, M, ldx, ws, ws_bytes, ARCHEAD_OP_TOPK);
  if (st != ARCHEAD_OK || M == 0) return st;
  if (!idx) return fail(ARCHEAD_E_INVALID_ARG, "idx is required");
  if (ldk < k) return fail(ARCHEAD_E_INVALID_ARG, "ldk < k");
  if (!aligned(idx, 8) || (vals && !aligned(vals, 4)))
    return fail(ARCHEAD_E_MISALIGNED, "idx / vals misaligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const WsLayout w = ws_layout(h, M, ARCHEAD_OP_TOPK);
  char* base = static_cast<char*>(ws);
  float* pv = reinterpret_cast<float*>(base + w.tk_pv_off);
  int* pi = reinterpret_cast<int*>(base + w.tk_pi_off);
  int64_t np = w.n_part;
  hipError_t e;
  if (w.tk_fused) {
    GemvArgs a = gemv_args(h, x, ldx, reinterpret_cast<uint64_t*>(base + w.tst_off));
    a.tk_val = pv;
    a.tk_idx = pi;
    a.tk_k = k;
    a.n_part = np;
    st = launch_gemv_passes(h, a, 1, false, np, s, true);
    if (st != ARCHEAD_OK) return st;
    void* margs[] = {&pv, &pi, &np, &k, &vals, &idx, &ldk};
    e = launch_topk_merge(np, k, 1, margs, s);
    return e == hipSuccess ? ARCHEAD_OK : hip_fail(e, "top-k merge launch");
  }
  const int64_t V = h->desc.V;
  float* lg = reinterpret_cast<float*>(base + w.tk_lg_off);
  // slices of whole 64-logit steps
  int64_t slice = (V + np - 1) / np;
  slice = (slice + 63) / 64 * 64;
  for (int64_t m0 = 0; m0 < M; m0 += w.tk_chunk) {
    const int64_t mc = M - m0 < w.tk_chunk ? M - m0 : w.tk_chunk;
    st = logits_run(h, static_cast<const uint16_t*>(x) + m0 * ldx, mc, ldx, lg, ARCHEAD_F32, V,
                    base + w.tk_in_off, s, w.tk_path);
    if (st != ARCHEAD_OK) return st;
    int64_t ldl = V;
    void* rargs[] = {&lg, &ldl, const_cast<int64_t*>(&V), &k, &slice, &pv, &pi};
    e = hipLaunchKernel(kern::topk_rows(), dim3(unsigned(np), unsigned(mc)), dim3(kBlock), rargs,
                        0, s);
    if (e != hipSuccess) return hip_fail(e, "top-k rows launch");
    float* vo = vals ? vals + m0 * ldk : nullptr;
    int64_t* io = idx + m0 * ldk;
    void* margs[] = {&pv, &pi, &np, &k, &vo, &io, &ldk};
    e = launch_topk_merge(np, k, mc, margs, s);
    if (e != hipSuccess) return hip_fail(e, "top-k merge launch");
  }
  return ARCHEAD_OK;
}

}  // extern "C"
