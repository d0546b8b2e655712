// Logit fidelity of the packed head to a dense reference head (Section 4,
// "Logit Fidelity", Table 8): per position, KL(p_ref || p_test), the summed
// squared logit error and the rank of the reference's top-1 token among the
// test logits, from which top-k agreement follows for every k.
//
// Each position's two fp32 logit rows are cut into chunks of kFChunk
// elements, one workgroup per (position, chunk), so that even one position
// spreads over the whole chip:
//   k_fid_part   per chunk: both maxima, the reference's first argmax, and
//                the softmax sums, p-weighted difference sum and squared
//                error relative to the chunk's own maxima (a second walk
//                over the chunk, from cache);
//   k_fid_merge  per position: the chunk partials in chunk order, rescaled
//                to the row maxima (fp64), give KL, the squared error and
//                the argmax; it also reads the test logit at the argmax and
//                clears the rank;
//   k_fid_rank   per chunk: test logits ranked ahead of that one (larger,
//                or equal at a smaller index), added to the rank with an
//                integer atomic (order-independent, so reproducible).
// Rows that start on 16-byte boundaries are read 16 bytes per lane.  It is
// an evaluation pass over logits already written (12 V bytes per position
// from memory), not part of the head's forward.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "internal.h"

using archead::fail;

namespace {

constexpr int kFBlock = 256;                 // threads per chunk
constexpr int kFWaves = kFBlock / 64;
constexpr int64_t kFChunk = 8192;            // elements per chunk (32 per thread)

struct FidPart {                             // one chunk's statistics
  float ma, mb;                              // chunk maxima of ref and test
  int64_t ia;                                // first index of ma (V if none)
  double sa, sb, t, sq;                      // relative to ma, mb
};

struct FidArgs {
  const float* ref;
  const float* test;
  int64_t ld_ref, ld_test, V, n_chunk;
  FidPart* part;                             // [M][n_chunk]
  float* bstar;                              // [M] test logit at the argmax
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

// Calls f(x, y, v) for the chunk's elements of this thread in increasing v:
// its 16-byte slots, then its elements of the ragged tail.
template <class F>
__device__ __forceinline__ void walk_chunk(const float* ra, const float* rb, int64_t lo,
                                           int64_t hi, bool vec, int tid, F&& f) {
  int64_t vend = lo;
  if (vec) {
    const int64_t ns = (hi - lo) / 4;
    vend = lo + 4 * ns;
    const float4* va = reinterpret_cast<const float4*>(ra + lo);
    const float4* vb = reinterpret_cast<const float4*>(rb + lo);
    int64_t j = tid;
    for (; j + kFBlock < ns; j += 2 * kFBlock) {
      const float4 x0 = va[j], y0 = vb[j], x1 = va[j + kFBlock], y1 = vb[j + kFBlock];
      const int64_t v0 = lo + 4 * j, v1 = lo + 4 * (j + kFBlock);
      f(x0.x, y0.x, v0); f(x0.y, y0.y, v0 + 1); f(x0.z, y0.z, v0 + 2); f(x0.w, y0.w, v0 + 3);
      f(x1.x, y1.x, v1); f(x1.y, y1.y, v1 + 1); f(x1.z, y1.z, v1 + 2); f(x1.w, y1.w, v1 + 3);
    }
    if (j < ns) {
      const float4 x0 = va[j], y0 = vb[j];
      const int64_t v0 = lo + 4 * j;
      f(x0.x, y0.x, v0); f(x0.y, y0.y, v0 + 1); f(x0.z, y0.z, v0 + 2); f(x0.w, y0.w, v0 + 3);
    }
  }
  for (int64_t v = vend + tid; v < hi; v += kFBlock) f(ra[v], rb[v], v);
}

// The same order over one row.
template <class F>
__device__ __forceinline__ void walk_row(const float* rb, int64_t lo, int64_t hi, bool vec,
                                         int tid, F&& f) {
  int64_t vend = lo;
  if (vec) {
    const int64_t ns = (hi - lo) / 4;
    vend = lo + 4 * ns;
    const float4* vb = reinterpret_cast<const float4*>(rb + lo);
    int64_t j = tid;
    for (; j + kFBlock < ns; j += 2 * kFBlock) {
      const float4 y0 = vb[j], y1 = vb[j + kFBlock];
      const int64_t v0 = lo + 4 * j, v1 = lo + 4 * (j + kFBlock);
      f(y0.x, v0); f(y0.y, v0 + 1); f(y0.z, v0 + 2); f(y0.w, v0 + 3);
      f(y1.x, v1); f(y1.y, v1 + 1); f(y1.z, v1 + 2); f(y1.w, v1 + 3);
    }
    if (j < ns) {
      const float4 y0 = vb[j];
      const int64_t v0 = lo + 4 * j;
      f(y0.x, v0); f(y0.y, v0 + 1); f(y0.z, v0 + 2); f(y0.w, v0 + 3);
    }
  }
  for (int64_t v = vend + tid; v < hi; v += kFBlock) f(rb[v], v);
}

__device__ __forceinline__ bool rows_vec(const float* ra, const float* rb) {
  return (reinterpret_cast<uintptr_t>(ra) % 16 == 0) && (reinterpret_cast<uintptr_t>(rb) % 16 == 0);
}

__global__ __launch_bounds__(kFBlock) void k_fid_part(FidArgs a) {
  __shared__ float s_f[kFWaves][2];
  __shared__ int64_t s_i[kFWaves];
  __shared__ double s_d[kFWaves][4];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t c = blockIdx.x, m = blockIdx.y;
  const float* ra = a.ref + m * a.ld_ref;
  const float* rb = a.test + m * a.ld_test;
  const int64_t lo = c * kFChunk, hi = lo + kFChunk < a.V ? lo + kFChunk : a.V;
  const bool vec = rows_vec(ra, rb);

  float ma = -INFINITY, mb = -INFINITY;
  int64_t ia = a.V;
  walk_chunk(ra, rb, lo, hi, vec, tid, [&](float x, float y, int64_t v) {
    if (x > ma) {   // strict: a thread keeps its first maximum
      ma = x;
      ia = v;
    }
    mb = fmaxf(mb, y);
  });
  for (int o = 32; o >= 1; o >>= 1) {
    max_first(ma, ia, __shfl_xor(ma, o), __shfl_xor(ia, o));
    mb = fmaxf(mb, __shfl_xor(mb, o));
  }
  if (lane == 0) {
    s_f[wv][0] = ma;
    s_f[wv][1] = mb;
    s_i[wv] = ia;
  }
  __syncthreads();
  ma = s_f[0][0];
  mb = s_f[0][1];
  ia = s_i[0];
  for (int w = 1; w < kFWaves; ++w) {
    max_first(ma, ia, s_f[w][0], s_i[w]);
    mb = fmaxf(mb, s_f[w][1]);
  }

  double sa = 0.0, sb = 0.0, t = 0.0, sq = 0.0;
  walk_chunk(ra, rb, lo, hi, vec, tid, [&](float x, float y, int64_t) {
    const float ea = expf(x - ma);
    const double diff = double(x) - double(y);
    sa += ea;
    sb += expf(y - mb);
    t += double(ea) * diff;
    sq += diff * diff;
  });
  for (int o = 32; o >= 1; o >>= 1) {
    sa += __shfl_xor(sa, o);
    sb += __shfl_xor(sb, o);
    t += __shfl_xor(t, o);
    sq += __shfl_xor(sq, o);
  }
  if (lane == 0) {
    s_d[wv][0] = sa;
    s_d[wv][1] = sb;
    s_d[wv][2] = t;
    s_d[wv][3] = sq;
  }
  __syncthreads();
  if (tid == 0) {
    FidPart p;
    p.ma = ma;
    p.mb = mb;
    p.ia = ia;
    p.sa = p.sb = p.t = p.sq = 0.0;
    for (int w = 0; w < kFWaves; ++w) {   // fixed order: reproducible
      p.sa += s_d[w][0];
      p.sb += s_d[w][1];
      p.t += s_d[w][2];
      p.sq += s_d[w][3];
    }
    a.part[m * a.n_chunk + c] = p;
  }
}

// one thread per position: the chunk partials in chunk order
__global__ void k_fid_merge(FidArgs a, int64_t M) {
  const int64_t m = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (m >= M) return;
  const FidPart* p = a.part + m * a.n_chunk;
  float ma = -INFINITY, mb = -INFINITY;
  int64_t ia = a.V;
  for (int64_t c = 0; c < a.n_chunk; ++c) {
    max_first(ma, ia, p[c].ma, p[c].ia);
    mb = fmaxf(mb, p[c].mb);
  }
  double sa = 0.0, sb = 0.0, t = 0.0, sq = 0.0;
  for (int64_t c = 0; c < a.n_chunk; ++c) {
    // a chunk's sums were taken relative to its own maxima
    const double fa = exp(double(p[c].ma) - double(ma));
    const double fb = exp(double(p[c].mb) - double(mb));
    sa += p[c].sa * fa;
    t += p[c].t * fa;
    sb += p[c].sb * fb;
    sq += p[c].sq;
  }
  if (ia >= a.V) ia = 0;   // no finite maximum: keep the index in range
  // sum_v p (log p - log q) with log p = a - ma - ln sa and
  // log q = b - mb - ln sb: E_p[a - b] + (mb - ma) + ln(sb / sa)
  a.kl[m] = float(t / sa + (double(mb) - double(ma)) + (log(sb) - log(sa)));
  a.sq[m] = float(sq);
  a.ref_idx[m] = ia;
  a.bstar[m] = a.test[m * a.ld_test + ia];
  a.rank[m] = 0;
}

__global__ __launch_bounds__(kFBlock) void k_fid_rank(FidArgs a) {
  __shared__ int64_t s_c[kFWaves];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t c = blockIdx.x, m = blockIdx.y;
  const float* rb = a.test + m * a.ld_test;
  const int64_t lo = c * kFChunk, hi = lo + kFChunk < a.V ? lo + kFChunk : a.V;
  const float bs = a.bstar[m];
  const int64_t ia = a.ref_idx[m];
  const bool vec = reinterpret_cast<uintptr_t>(rb) % 16 == 0;
  int64_t cnt = 0;
  walk_row(rb, lo, hi, vec, tid, [&](float y, int64_t v) {
    cnt += (y > bs || (y == bs && v < ia)) ? 1 : 0;
  });
  for (int o = 32; o >= 1; o >>= 1) cnt += __shfl_xor(cnt, o);
  if (lane == 0) s_c[wv] = cnt;
  __syncthreads();
  if (tid == 0) {
    int64_t tot = 0;
    for (int w = 0; w < kFWaves; ++w) tot += s_c[w];
    if (tot) atomicAdd(reinterpret_cast<unsigned long long*>(a.rank + m), (unsigned long long)tot);
  }
}

bool aligned(const void* p, uintptr_t n) { return (reinterpret_cast<uintptr_t>(p) % n) == 0; }

size_t fid_ws(int64_t M, int64_t V, int64_t* n_chunk, size_t* bstar_off) {
  const int64_t nc = (V + kFChunk - 1) / kFChunk;
  const size_t part = size_t(M) * size_t(nc) * sizeof(FidPart);
  const size_t boff = (part + 255) & ~size_t(255);
  if (n_chunk) *n_chunk = nc;
  if (bstar_off) *bstar_off = boff;
  return boff + size_t(M) * 4;
}

}  // namespace

extern "C" {

size_t archead_fidelity_workspace_bytes(int64_t M, int64_t V) {
  if (M <= 0 || V < 1 || M > INT32_MAX || V > INT32_MAX) return 0;
  return fid_ws(M, V, nullptr, nullptr);
}

archead_status archead_logit_fidelity(const float* ref, int64_t ld_ref, const float* test,
                                      int64_t ld_test, int64_t M, int64_t V, float* kl,
                                      float* sq, int64_t* ref_idx, int64_t* rank, void* ws,
                                      size_t ws_bytes, void* stream) {
  archead::clear_error();
  if (M < 0 || M > 65535) return fail(ARCHEAD_E_INVALID_ARG, "M = %lld out of range", (long long)M);
  if (V < 1 || V > INT32_MAX) return fail(ARCHEAD_E_INVALID_ARG, "V = %lld out of range", (long long)V);
  if (M == 0) return ARCHEAD_OK;
  if (ld_ref < V || ld_test < V)
    return fail(ARCHEAD_E_INVALID_ARG, "leading dimensions must be >= V");
  if (!ref || !test || !kl || !sq || !ref_idx || !rank || !ws)
    return fail(ARCHEAD_E_INVALID_ARG, "null pointer");
  if (!aligned(ref, 4) || !aligned(test, 4) || !aligned(kl, 4) || !aligned(sq, 4) ||
      !aligned(ref_idx, 8) || !aligned(rank, 8) || !aligned(ws, 256))
    return fail(ARCHEAD_E_MISALIGNED, "misaligned pointer");
  int64_t nc = 0;
  size_t boff = 0;
  const size_t need = fid_ws(M, V, &nc, &boff);
  if (ws_bytes < need)
    return fail(ARCHEAD_E_WORKSPACE, "workspace of %zu bytes, %zu needed", ws_bytes, need);
  FidArgs a{ref, test, ld_ref, ld_test, V, nc, static_cast<FidPart*>(ws),
            reinterpret_cast<float*>(static_cast<char*>(ws) + boff), kl, sq, ref_idx, rank};
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid{unsigned(nc), unsigned(M), 1u};
  hipLaunchKernelGGL(k_fid_part, grid, dim3(kFBlock), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) {
    hipLaunchKernelGGL(k_fid_merge, dim3(unsigned((M + 63) / 64)), dim3(64), 0, s, a, M);
    e = hipGetLastError();
  }
  if (e == hipSuccess) {
    hipLaunchKernelGGL(k_fid_rank, grid, dim3(kFBlock), 0, s, a);
    e = hipGetLastError();
  }
  if (e != hipSuccess)
    return fail(ARCHEAD_E_HIP, "fidelity launch: %s", hipGetErrorString(e));
  return ARCHEAD_OK;
}

}  // extern "C"
