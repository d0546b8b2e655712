// Logit fidelity of the packed head to a dense reference head (Section 4,
// "Logit Fidelity", Table 8): per position, KL(p_ref || p_test), the summed
// squared logit error and the rank of the reference's top-1 token among the
// test logits, from which top-k agreement follows for every k.
//
// One workgroup per position walks the two fp32 logit rows twice: first for
// both row maxima and the reference's first argmax, then for the softmax
// sums, the KL numerator, the squared error and the rank count.  Rows whose
// starts are 16-byte aligned are read 16 bytes per lane, two loads per row
// in flight per lane, then the ragged tail element by element.  It is an
// evaluation pass over logits that are already written (2 x 4 V bytes per
// position, the second walk mostly from the last-level caches), not part of
// the head's forward.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "internal.h"

using archead::fail;

namespace {

constexpr int kFBlock = 512;                 // threads per position
constexpr int kFWaves = kFBlock / 64;

struct FidArgs {
  const float* ref;
  const float* test;
  int64_t ld_ref, ld_test, V;
  float* kl;
  float* sq;
  int64_t* ref_idx;
  int64_t* rank;
};

// (value, index) with the larger value winning and the smaller index on ties
__device__ __forceinline__ void max_first(float& v, int64_t& i, float ov, int64_t oi) {
  if (ov > v || (ov == v && oi < i)) {
    v = ov;
    i = oi;
  }
}

__global__ __launch_bounds__(kFBlock) void k_fidelity(FidArgs a) {
  __shared__ float s_f[kFWaves][2];
  __shared__ int64_t s_i[kFWaves];
  __shared__ double s_d[kFWaves][4];
  __shared__ int64_t s_c[kFWaves];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t m = blockIdx.x;
  const float* ra = a.ref + m * a.ld_ref;
  const float* rb = a.test + m * a.ld_test;
  const int64_t V = a.V;

  // walk 1: max of ref with its first index, max of test.  Each thread
  // visits its indices in increasing order (its 16-byte slots, then its
  // tail elements), so a strict comparison keeps its first maximum.
  float amax = -INFINITY, bmax = -INFINITY;
  int64_t aidx = V;
  const bool vec = (reinterpret_cast<uintptr_t>(ra) % 16 == 0) &&
                   (reinterpret_cast<uintptr_t>(rb) % 16 == 0);
  const int64_t nv = vec ? V / 4 : 0;   // float4 slots; elements 4 nv .. V - 1 follow
  auto walk = [&](auto&& f) {
    const float4* va = reinterpret_cast<const float4*>(ra);
    const float4* vb = reinterpret_cast<const float4*>(rb);
    int64_t j = tid;
    for (; j + kFBlock < nv; j += 2 * kFBlock) {
      const float4 x0 = va[j], y0 = vb[j], x1 = va[j + kFBlock], y1 = vb[j + kFBlock];
      f(x0.x, y0.x, 4 * j); f(x0.y, y0.y, 4 * j + 1); f(x0.z, y0.z, 4 * j + 2); f(x0.w, y0.w, 4 * j + 3);
      const int64_t v1 = 4 * (j + kFBlock);
      f(x1.x, y1.x, v1); f(x1.y, y1.y, v1 + 1); f(x1.z, y1.z, v1 + 2); f(x1.w, y1.w, v1 + 3);
    }
    if (j < nv) {
      const float4 x0 = va[j], y0 = vb[j];
      f(x0.x, y0.x, 4 * j); f(x0.y, y0.y, 4 * j + 1); f(x0.z, y0.z, 4 * j + 2); f(x0.w, y0.w, 4 * j + 3);
    }
    for (int64_t v = 4 * nv + tid; v < V; v += kFBlock) f(ra[v], rb[v], v);
  };
  // each thread visits its indices in increasing order
  walk([&](float x, float y, int64_t v) {
    if (x > amax) {
      amax = x;
      aidx = v;
    }
    bmax = fmaxf(bmax, y);
  });
  for (int o = 32; o >= 1; o >>= 1) {
    max_first(amax, aidx, __shfl_xor(amax, o), __shfl_xor(aidx, o));
    bmax = fmaxf(bmax, __shfl_xor(bmax, o));
  }
  if (lane == 0) {
    s_f[wv][0] = amax;
    s_f[wv][1] = bmax;
    s_i[wv] = aidx;
  }
  __syncthreads();
  amax = s_f[0][0];
  bmax = s_f[0][1];
  aidx = s_i[0];
  for (int w = 1; w < kFWaves; ++w) {
    max_first(amax, aidx, s_f[w][0], s_i[w]);
    bmax = fmaxf(bmax, s_f[w][1]);
  }
  if (aidx >= V) aidx = 0;   // no finite maximum: keep the index in range
  const float bstar = rb[aidx];

  // walk 2: softmax sums of both rows, sum of p-weighted differences,
  // squared error, and the count of test logits ranked ahead of the
  // reference's top-1 token (larger, or equal at a smaller index)
  double sa = 0.0, sb = 0.0, t = 0.0, sq = 0.0;
  int64_t cnt = 0;
  walk([&](float x, float y, int64_t v) {
    const float ea = expf(x - amax);
    const double diff = double(x) - double(y);
    sa += ea;
    sb += expf(y - bmax);
    t += double(ea) * diff;
    sq += diff * diff;
    cnt += (y > bstar || (y == bstar && v < aidx)) ? 1 : 0;
  });
  for (int o = 32; o >= 1; o >>= 1) {
    sa += __shfl_xor(sa, o);
    sb += __shfl_xor(sb, o);
    t += __shfl_xor(t, o);
    sq += __shfl_xor(sq, o);
    cnt += __shfl_xor(cnt, o);
  }
  if (lane == 0) {
    s_d[wv][0] = sa;
    s_d[wv][1] = sb;
    s_d[wv][2] = t;
    s_d[wv][3] = sq;
    s_c[wv] = cnt;
  }
  __syncthreads();
  if (tid == 0) {
    sa = sb = t = sq = 0.0;
    cnt = 0;
    for (int w = 0; w < kFWaves; ++w) {   // fixed order: reproducible
      sa += s_d[w][0];
      sb += s_d[w][1];
      t += s_d[w][2];
      sq += s_d[w][3];
      cnt += s_c[w];
    }
    // sum_v p (log p - log q) with log p = a - amax - ln sa and
    // log q = b - bmax - ln sb: E_p[a - b] + (bmax - amax) + ln(sb / sa)
    const double kl = t / sa + (double(bmax) - double(amax)) + (log(sb) - log(sa));
    a.kl[m] = float(kl);
    a.sq[m] = float(sq);
    a.ref_idx[m] = aidx;
    a.rank[m] = cnt;
  }
}

bool aligned(const void* p, uintptr_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

}  // namespace

extern "C" {

archead_status archead_logit_fidelity(const float* ref, int64_t ld_ref, const float* test,
                                      int64_t ld_test, int64_t M, int64_t V, float* kl,
                                      float* sq, int64_t* ref_idx, int64_t* rank,
                                      void* stream) {
  archead::clear_error();
  if (M < 0 || M > INT32_MAX) return fail(ARCHEAD_E_INVALID_ARG, "M = %lld out of range", (long long)M);
  if (V < 1 || V > INT32_MAX) return fail(ARCHEAD_E_INVALID_ARG, "V = %lld out of range", (long long)V);
  if (M == 0) return ARCHEAD_OK;
  if (ld_ref < V || ld_test < V)
    return fail(ARCHEAD_E_INVALID_ARG, "leading dimensions must be >= V");
  if (!ref || !test || !kl || !sq || !ref_idx || !rank)
    return fail(ARCHEAD_E_INVALID_ARG, "null pointer");
  if (!aligned(ref, 4) || !aligned(test, 4) || !aligned(kl, 4) || !aligned(sq, 4) ||
      !aligned(ref_idx, 8) || !aligned(rank, 8))
    return fail(ARCHEAD_E_MISALIGNED, "misaligned pointer");
  FidArgs a{ref, test, ld_ref, ld_test, V, kl, sq, ref_idx, rank};
  hipLaunchKernelGGL(k_fidelity, dim3(unsigned(M)), dim3(kFBlock), 0,
                     static_cast<hipStream_t>(stream), a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return fail(ARCHEAD_E_HIP, "fidelity launch: %s", hipGetErrorString(e));
  return ARCHEAD_OK;
}

}  // extern "C"
