// Top-k selection: the single-token decode GEMV with the fused top-k
// epilogue, the top-k of rows of fp32 logits, and the merge of per-partial
// lists.  Every list is in the order of the first-index argmax (larger value
// first, equal values by smaller index), so the merged result is the first k
// entries of the stable descending sort of the token's logits.
#include "dev_gemv.cuh"
#include "kernels.h"

namespace {

using GemvFn = void (*)(GemvArgs);

template <bool SC8, int GEN>
GemvFn gemv_topk_by_lpr(int lpr) {
  if constexpr (GEN > 0) {
    switch (lpr) {
      case 8: return k_gemv<1, 8, false, SC8, GEN, true>;
      case 16: return k_gemv<1, 16, false, SC8, GEN, true>;
      default: return nullptr;
    }
  } else {
    switch (lpr) {
      case 1: return k_gemv<1, 1, false, SC8, GEN, true>;
      case 2: return k_gemv<1, 2, false, SC8, GEN, true>;
      case 4: return k_gemv<1, 4, false, SC8, GEN, true>;
      case 8: return k_gemv<1, 8, false, SC8, GEN, true>;
      case 16: return k_gemv<1, 16, false, SC8, GEN, true>;
      case 32: return k_gemv<1, 32, false, SC8, GEN, true>;
      default: return k_gemv<1, 64, false, SC8, GEN, true>;
    }
  }
}

template <int GEN>
const void* gemv_topk_fn(int lpr, bool sc8) {
  GemvFn fn = sc8 ? gemv_topk_by_lpr<true, GEN>(lpr) : gemv_topk_by_lpr<false, GEN>(lpr);
  return reinterpret_cast<const void*>(fn);
}

// Offer entries j in [lo, hi) of one wave's share of a flat array of
// candidates (value val(j), index idx(j)) to the wave's list: 64 per step,
// wave w of the workgroup taking steps lo + 64 w, lo + 64 (w + kWaves), ...;
// kScanBatch steps' loads are issued together before any is offered, so a
// scan costs one memory latency per batch, not per step.  Candidates ranked
// below the floor (fv, fi) are not offered.
constexpr int kScanBatch = 8;
template <typename Val, typename Idx>
__device__ __forceinline__ void tk_scan(int64_t lo, int64_t hi, Val val, Idx idx, int lane, int wid,
                                        int k, float& lv, int& li, float& bv, int& bi,
                                        float fv = -INFINITY, int fi = kNoIdx) {
  for (int64_t b = lo + int64_t(wid) * 64; b < hi; b += int64_t(kScanBatch) * kBlock) {
    float cv[kScanBatch];
    int ci[kScanBatch];
#pragma unroll
    for (int u = 0; u < kScanBatch; ++u) {
      const int64_t j = b + int64_t(u) * kBlock + lane;
      cv[u] = j < hi ? val(j) : -INFINITY;
      ci[u] = j < hi ? idx(j) : kNoIdx;
    }
#pragma unroll
    for (int u = 0; u < kScanBatch; ++u)
      tk_offer(lv, li, bv, bi, cv[u], ci[u],
               (b + int64_t(u) * kBlock + lane < hi) & !tk_better(fv, fi, cv[u], ci[u]), lane, k);
  }
}

__device__ __forceinline__ void tk_pick(float& bv, int& bi, float ov, int oi) {
  const bool t = tk_better(ov, oi, bv, bi);
  bv = t ? ov : bv;
  bi = t ? oi : bi;
}
template <int CTRL>
__device__ __forceinline__ void tk_pick_dpp(float& v, int& i) {
  const float ov = dpp_swap<CTRL>(v);
  const int oi = __builtin_amdgcn_update_dpp(0, i, CTRL, 0xF, 0xF, false);
  tk_pick(v, i, ov, oi);
}
// the best pair of each row of 16 lanes, in every lane of the row
__device__ __forceinline__ void tk_row16_best(float& v, int& i) {
  tk_pick_dpp<0xB1>(v, i);
  tk_pick_dpp<0x4E>(v, i);
  tk_pick_dpp<0x141>(v, i);
  tk_pick_dpp<0x140>(v, i);
}

// Per (partial p, token m) of grid (n_part, M): the k best pairs of
// logits[m, v] over the slice v in [p * slice, min(V, (p + 1) * slice)),
// into pv / pi [M][n_part][k].
//  * For k <= 16, a floor first: each lane's best logit of the slice (its
//    share: v = lo + tid, lo + tid + kBlock, ...), then k rounds of the
//    wave's best among those (the owner drops it after each): the k-th is
//    ranked at or below the wave's own k-th best (k lanes hold one at least
//    as good), so the wave's list only sees candidates at or above it.
//  * The four wave lists then merge by rank (distinct indices: every entry
//    has a distinct rank), not by inserting one list into another.
__global__ __launch_bounds__(kBlock) void k_topk_rows(const float* logits, int64_t ldl, int64_t V,
                                                      int k, int64_t slice, float* pv, int* pi) {
  __shared__ float sv[kWaves * 64];
  __shared__ int si[kWaves * 64];
  __shared__ float ov[kTopKMax];
  __shared__ int oi[kTopKMax];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int64_t m = blockIdx.y, p = blockIdx.x, n_part = gridDim.x;
  const int64_t lo = p * slice;
  const int64_t hi = lo + slice < V ? lo + slice : V;
  const float* row = logits + m * ldl;
  float fv = -INFINITY;
  int fi = kNoIdx;
  if (k <= 16) {
    float cv = -INFINITY;
    int ci = kNoIdx;
    for (int64_t j0 = lo + tid; j0 < hi; j0 += int64_t(kScanBatch) * kBlock) {
      float v[kScanBatch];
#pragma unroll
      for (int u = 0; u < kScanBatch; ++u) {
        const int64_t j = j0 + int64_t(u) * kBlock;
        v[u] = j < hi ? row[j] : -INFINITY;
      }
#pragma unroll
      for (int u = 0; u < kScanBatch; ++u) {
        const int64_t j = j0 + int64_t(u) * kBlock;
        if (j < hi) tk_pick(cv, ci, v[u], int(j));
      }
    }
    for (int r = 0; r < k; ++r) {
      float gv = cv;
      int gi = ci;
      tk_row16_best(gv, gi);
      float bv = rlane_f(gv, 0);
      int bi = __builtin_amdgcn_readlane(gi, 0);
#pragma unroll
      for (int rr = 1; rr < 4; ++rr)
        tk_pick(bv, bi, rlane_f(gv, 16 * rr), __builtin_amdgcn_readlane(gi, 16 * rr));
      fv = bv;
      fi = bi;
      if (bi != kNoIdx && ci == bi) {
        cv = -INFINITY;
        ci = kNoIdx;
      }
    }
  }
  float lv = -INFINITY, bv = -INFINITY;
  int li = kNoIdx, bi = kNoIdx;
  tk_scan(lo, hi, [&](int64_t j) { return row[j]; }, [&](int64_t j) { return int(j); }, lane, wid,
          k, lv, li, bv, bi, fv, fi);
  tk_rank_merge<kWaves>(lv, li, tid, k, sv, si, ov, oi);
  if (tid < k) {
    const int64_t o = (m * n_part + p) * k + tid;
    pv[o] = ov[tid];
    pi[o] = oi[tid];
  }
}

// Per token m (grid M, workgroups of kBlock): the k best of its n_part partial
// lists of k pairs (scanned as one flat array of n_part * k candidates), out to
// vals[m * ldk + j] (may be null) and idx[m * ldk + j], j < k; a slot no
// value reached (fewer than k non-NaN logits) gets (-inf, -1).
__global__ __launch_bounds__(kBlock) void k_topk_merge_scan(const float* pv, const int* pi,
                                                       int64_t n_part, int k, float* vals,
                                                       int64_t* idx, int64_t ldk) {
  __shared__ float sv[kWaves * 64];
  __shared__ int si[kWaves * 64];
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int64_t m = blockIdx.x;
  const float* v = pv + m * n_part * k;
  const int* ix = pi + m * n_part * k;
  // a floor for the result's k-th entry: each list holds k entries ranked at
  // or above its own k-th, so the best of the lists' k-th entries is ranked
  // at or below the final k-th; candidates ranked below it are skipped
  float fv = -INFINITY;
  int fi = kNoIdx;
  for (int64_t p = threadIdx.x; p < n_part; p += kBlock) {
    const float c = v[p * k + k - 1];
    const int ci = ix[p * k + k - 1];
    if (tk_better(c, ci, fv, fi)) { fv = c; fi = ci; }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float ov = __shfl_xor(fv, off, 64);
    const int oi = __shfl_xor(fi, off, 64);
    if (tk_better(ov, oi, fv, fi)) { fv = ov; fi = oi; }
  }
  if (lane == 0) { sv[wid] = fv; si[wid] = fi; }
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kWaves; ++w)
    if (tk_better(sv[w], si[w], fv, fi)) { fv = sv[w]; fi = si[w]; }
  __syncthreads();
  float lv = -INFINITY, bv = -INFINITY;
  int li = kNoIdx, bi = kNoIdx;
  tk_scan(0, n_part * k, [&](int64_t j) { return v[j]; }, [&](int64_t j) { return ix[j]; }, lane,
          wid, k, lv, li, bv, bi, fv, fi);
  tk_block_merge<kWaves>(lv, li, bv, bi, lane, wid, k, sv, si);
  if (wid == 0 && lane < k) {
    if (vals) vals[m * ldk + lane] = lv;
    idx[m * ldk + lane] = li == kNoIdx ? int64_t(-1) : int64_t(li);
  }
}

// Per token m (grid M, workgroups of kMergeBlock), for at most kMergeBlock *
// kMergeC candidates: the same result in k rounds.  Each thread holds up to
// kMergeC candidates and its best one; a round finds the best of the
// workgroup (DPP within rows of 16 lanes, then the four rows of the wave,
// then the waves through LDS), writes it out, and its owner (indices are
// distinct across the partial lists) drops it and takes its next best.  The
// cost is k rounds, whatever the values.
constexpr int kMergeC = 8;
static_assert(archead::kTopKMergeBlock == 1024 && kMergeC == archead::kTopKMergeC,
              "host and kernel agree on the merge workgroup");

template <int kMergeBlock>
__global__ __launch_bounds__(kMergeBlock) void k_topk_merge(const float* pv, const int* pi,
                                                            int64_t n_part, int k, float* vals,
                                                            int64_t* idx, int64_t ldk) {
  constexpr int kMergeWaves = kMergeBlock / 64;
  __shared__ float wv[2][kMergeWaves];
  __shared__ int wi[2][kMergeWaves];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t m = blockIdx.x;
  const int64_t n = n_part * k;
  const float* v = pv + m * n;
  const int* ix = pi + m * n;
  float cv[kMergeC];
  int ci[kMergeC];
#pragma unroll
  for (int u = 0; u < kMergeC; ++u) {
    const int64_t j = int64_t(u) * kMergeBlock + tid;
    cv[u] = j < n ? v[j] : -INFINITY;
    ci[u] = j < n ? ix[j] : kNoIdx;
  }
  float tv = -INFINITY;
  int ti = kNoIdx;
#pragma unroll
  for (int u = 0; u < kMergeC; ++u) tk_pick(tv, ti, cv[u], ci[u]);
  for (int r = 0; r < k; ++r) {
    float bv = tv;
    int bi = ti;
    tk_row16_best(bv, bi);
    float gv = rlane_f(bv, 0);
    int gi = __builtin_amdgcn_readlane(bi, 0);
#pragma unroll
    for (int row = 1; row < 4; ++row)
      tk_pick(gv, gi, rlane_f(bv, 16 * row), __builtin_amdgcn_readlane(bi, 16 * row));
    if (lane == 0) {
      wv[r & 1][wid] = gv;
      wi[r & 1][wid] = gi;
    }
    __syncthreads();
    gv = lane < kMergeWaves ? wv[r & 1][lane] : -INFINITY;
    gi = lane < kMergeWaves ? wi[r & 1][lane] : kNoIdx;
    tk_row16_best(gv, gi);
    gv = rlane_f(gv, 0);
    gi = __builtin_amdgcn_readlane(gi, 0);
    if (tid == 0) {
      if (vals) vals[m * ldk + r] = gv;
      idx[m * ldk + r] = gi == kNoIdx ? int64_t(-1) : int64_t(gi);
    }
    if (gi != kNoIdx && ti == gi) {
#pragma unroll
      for (int u = 0; u < kMergeC; ++u) {
        const bool hit = ci[u] == gi;
        cv[u] = hit ? -INFINITY : cv[u];
        ci[u] = hit ? kNoIdx : ci[u];
      }
      tv = -INFINITY;
      ti = kNoIdx;
#pragma unroll
      for (int u = 0; u < kMergeC; ++u) tk_pick(tv, ti, cv[u], ci[u]);
    }
  }
}

}  // namespace

namespace archead {
namespace kern {

const void* gemv_topk(int lpr, bool sc8, int gen) {
  if (gen == 2) return gemv_topk_fn<2>(lpr, sc8);
  if (gen == 1) return gemv_topk_fn<1>(lpr, sc8);
  return gemv_topk_fn<0>(lpr, sc8);
}

const void* topk_rows() { return reinterpret_cast<const void*>(k_topk_rows); }
const void* topk_merge(int block) {
  return block == 256 ? reinterpret_cast<const void*>(k_topk_merge<256>)
                      : reinterpret_cast<const void*>(k_topk_merge<1024>);
}
const void* topk_merge_scan() { return reinterpret_cast<const void*>(k_topk_merge_scan); }

}  // namespace kern
}  // namespace archead
