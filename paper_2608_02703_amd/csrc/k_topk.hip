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

// Per (partial p, token m) of grid (n_part, M): the k best pairs of
// logits[m, v] over the slice v in [p * slice, min(V, (p + 1) * slice)),
// into pv / pi [M][n_part][k].  Each wave reads 64 consecutive logits per
// step (coalesced), offers them to its list, and the four lists are merged.
__global__ __launch_bounds__(kBlock) void k_topk_rows(const float* logits, int64_t ldl, int64_t V,
                                                      int k, int64_t slice, float* pv, int* pi) {
  __shared__ float sv[kWaves * 64];
  __shared__ int si[kWaves * 64];
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int64_t m = blockIdx.y, p = blockIdx.x, n_part = gridDim.x;
  const int64_t lo = p * slice;
  const int64_t hi = lo + slice < V ? lo + slice : V;
  const float* row = logits + m * ldl;
  float lv = -INFINITY, bv = -INFINITY;
  int li = kNoIdx, bi = kNoIdx;
  for (int64_t b = lo + wid * 64; b < hi; b += kBlock) {
    const int64_t v = b + lane;
    const bool ok = v < hi;
    const float x = ok ? row[v] : -INFINITY;
    tk_offer(lv, li, bv, bi, x, int(v), ok, lane, k);
  }
  tk_block_merge<kWaves>(lv, li, bv, bi, lane, wid, k, sv, si);
  if (wid == 0 && lane < k) {
    const int64_t o = (m * n_part + p) * k + lane;
    pv[o] = lv;
    pi[o] = li;
  }
}

// Per token m (grid M): the k best of its n_part partial lists of k pairs,
// out to vals[m * ldk + j] (may be null) and idx[m * ldk + j], j < k; a slot
// no value reached (fewer than k non-NaN logits) gets (-inf, -1).
__global__ __launch_bounds__(kBlock) void k_topk_merge(const float* pv, const int* pi,
                                                       int64_t n_part, int k, float* vals,
                                                       int64_t* idx, int64_t ldk) {
  __shared__ float sv[kWaves * 64];
  __shared__ int si[kWaves * 64];
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int64_t m = blockIdx.x;
  float lv = -INFINITY, bv = -INFINITY;
  int li = kNoIdx, bi = kNoIdx;
  for (int64_t p = wid; p < n_part; p += kWaves) {
    const bool ok = lane < k;
    const int64_t o = (m * n_part + p) * k + lane;
    const float x = ok ? pv[o] : -INFINITY;
    const int i = ok ? pi[o] : kNoIdx;
    tk_offer(lv, li, bv, bi, x, i, ok, lane, k);
  }
  tk_block_merge<kWaves>(lv, li, bv, bi, lane, wid, k, sv, si);
  if (wid == 0 && lane < k) {
    if (vals) vals[m * ldk + lane] = lv;
    idx[m * ldk + lane] = li == kNoIdx ? int64_t(-1) : int64_t(li);
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
const void* topk_merge() { return reinterpret_cast<const void*>(k_topk_merge); }

}  // namespace kern
}  // namespace archead
