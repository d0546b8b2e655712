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
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "archead.h"
#include "internal.h"

namespace {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

constexpr int kBlock = 256;          // 4 waves of 64
constexpr int kWaves = kBlock / 64;
constexpr int kRowsPerStep = 8;      // rows (per lane segment) of one GEMV step
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}
__device__ __forceinline__ float f16_to_f32(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);
}
__device__ __forceinline__ float bf16_lo(uint32_t p) { return __uint_as_float(p << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t p) { return __uint_as_float(p & 0xffff0000u); }

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

// ------------------------------------------------------------------ stage 1
// t[m, k] = sum_i (s[k, i/grp] c[k, i]) x[m, i] for the rows k of V_c (k <
// r_c) then of B_w.  One wave per (k, block of 8 tokens); each lane covers
// 8 consecutive elements per step.  s * c is exact in fp32 (11 x 8 bits).
struct Stage1Args {
  const uint16_t* x;
  int64_t ldx, M, d;
  const int8_t* cv;
  const uint16_t* sv;
  int64_t gv, rc;
  const int8_t* cb;
  const uint16_t* sb;
  int64_t gb, rr;
  float* t;  // [M, rc + rr]
};

constexpr int kS1Tok = 8;

__global__ __launch_bounds__(kBlock) void k_stage1(Stage1Args a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = int64_t(blockIdx.x) * kWaves + (threadIdx.x >> 6);
  const int64_t R = a.rc + a.rr;
  const int64_t mblocks = (a.M + kS1Tok - 1) / kS1Tok;
  if (wave >= R * mblocks) return;  // uniform per wave
  const int64_t k = wave % R, m0 = (wave / R) * kS1Tok;
  const bool core = k < a.rc;
  const int8_t* crow = core ? a.cv + k * a.d : a.cb + (k - a.rc) * a.d;
  const int64_t grp = core ? a.gv : a.gb;
  const uint16_t* srow = core ? a.sv + k * (a.d / a.gv) : a.sb + (k - a.rc) * (a.d / a.gb);
  const int ntok = int(a.M - m0 < kS1Tok ? a.M - m0 : kS1Tok);
  float acc[kS1Tok];
#pragma unroll
  for (int j = 0; j < kS1Tok; ++j) acc[j] = 0.f;
  for (int64_t i = int64_t(lane) * 8; i < a.d; i += 512) {
    const uint2 cw = *reinterpret_cast<const uint2*>(crow + i);
    const float s = f16_to_f32(srow[i / grp]);
    float w[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      w[j] = float(int8_t(cw.x >> (8 * j))) * s;
      w[4 + j] = float(int8_t(cw.y >> (8 * j))) * s;
    }
#pragma unroll
    for (int tt = 0; tt < kS1Tok; ++tt) {
      if (tt < ntok) {
        const uint4 xv = *reinterpret_cast<const uint4*>(a.x + (m0 + tt) * a.ldx + i);
        const uint32_t xs[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[tt] = fmaf(bf16_lo(xs[j]), w[2 * j], acc[tt]);
          acc[tt] = fmaf(bf16_hi(xs[j]), w[2 * j + 1], acc[tt]);
        }
      }
    }
  }
#pragma unroll
  for (int tt = 0; tt < kS1Tok; ++tt) {
    const float s = seg_sum<64>(acc[tt]);
    if (lane == 0 && tt < ntok) a.t[(m0 + tt) * R + k] = s;
  }
}

// ------------------------------------------------------------ decode GEMV
// Lanes are split into segments of LPR lanes; a segment owns one vocabulary
// row at a time and walks along d in 16-byte chunks (32 codes), LPR chunks
// per iteration, so each segment load is LPR * 16 contiguous bytes.  A wave
// step covers kRowsPerStep rows per segment.  Waves get contiguous, balanced
// ranges of steps (persistent grid).  x, the chunk biases and t sit in LDS.
struct GemvArgs {
  const uint8_t* codes;
  const uint16_t* rs;
  const int8_t* cu;
  const uint16_t* su;
  const int8_t* ca;
  const uint16_t* sa;
  const uint16_t* x;
  int64_t ldx;
  const float* t;  // [M, rc + rr]
  int64_t tok0;    // first token of this pass
  int64_t V, d, g, rc, rr;
  int64_t nsteps;  // ceil(V / rows per wave step)
  int nit;         // iterations along d: (d / 32) / LPR
  void* out;
  int64_t ldo;
  int out_bf16;
  // fused CE
  const void* tgt;
  int tgt64;
  float2* part;    // [M, n_part]
  int64_t n_part;
  float* tgt_logit;  // [M]
};

template <int TOK, int LPR, bool CE>
__global__ __launch_bounds__(kBlock) void k_gemv(GemvArgs a) {
  constexpr int SEG = 64 / LPR;              // rows in flight per wave
  constexpr int RB = kRowsPerStep;
  constexpr int WR = RB * SEG;               // rows per wave step
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ float2 red[kWaves][TOK];

  const int64_t C = a.d / 32;                // 16-byte chunks per row
  const int64_t R = a.rc + a.rr;
  uint16_t* sx = reinterpret_cast<uint16_t*>(smem);          // [TOK][d]
  float* sxb = reinterpret_cast<float*>(sx + TOK * a.d);      // [TOK][C]
  float* st = sxb + TOK * C;                                  // [TOK][R]

  const int64_t x8 = a.d / 8;
  for (int64_t i = threadIdx.x; i < TOK * x8; i += kBlock) {
    const int64_t tt = i / x8, j = i - tt * x8;
    reinterpret_cast<uint4*>(sx)[i] =
        *reinterpret_cast<const uint4*>(a.x + (a.tok0 + tt) * a.ldx + j * 8);
  }
  for (int64_t i = threadIdx.x; i < TOK * R; i += kBlock) {
    const int64_t tt = i / R;
    st[i] = a.t[(a.tok0 + tt) * R + (i - tt * R)];
  }
  __syncthreads();
  for (int64_t i = threadIdx.x; i < TOK * C; i += kBlock) {
    const int64_t tt = i / C, c = i - tt * C;
    const uint32_t* p = reinterpret_cast<const uint32_t*>(sx + tt * a.d + c * 32);
    float s = 0.f;
    for (int j = 0; j < 16; ++j) s += bf16_lo(p[j]) + bf16_hi(p[j]);
    sxb[i] = -float(archead::kInt4Bias) * s;
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int seg = lane / LPR, sl = lane % LPR;
  const int64_t W = int64_t(gridDim.x) * kWaves;
  const int64_t gw = int64_t(blockIdx.x) * kWaves + wid;
  const int64_t s_begin = a.nsteps * gw / W, s_end = a.nsteps * (gw + 1) / W;
  const int64_t rowbytes = a.d / 2, ngrp = a.d / a.g;

  float mx[TOK], se[TOK];
#pragma unroll
  for (int tt = 0; tt < TOK; ++tt) { mx[tt] = -INFINITY; se[tt] = 0.f; }
  int64_t y[TOK];
  if constexpr (CE) {
#pragma unroll
    for (int tt = 0; tt < TOK; ++tt)
      y[tt] = a.tgt64 ? reinterpret_cast<const int64_t*>(a.tgt)[a.tok0 + tt]
                      : int64_t(reinterpret_cast<const int32_t*>(a.tgt)[a.tok0 + tt]);
  }

  for (int64_t step = s_begin; step < s_end; ++step) {
    float acc[RB][TOK];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int tt = 0; tt < TOK; ++tt) acc[rb][tt] = 0.f;
    const int64_t vbase = step * WR + seg;

    for (int it = 0; it < a.nit; ++it) {
      const int64_t c = int64_t(it) * LPR + sl;
      uint4 q[RB];
      uint16_t sc[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int64_t v = vbase + rb * SEG;
        if (v < a.V) {
          q[rb] = *reinterpret_cast<const uint4*>(a.codes + v * rowbytes + c * 16);
          sc[rb] = a.rs[v * ngrp + (c * 32) / a.g];
        } else {
          q[rb] = make_uint4(0x88888888u, 0x88888888u, 0x88888888u, 0x88888888u);
          sc[rb] = 0;
        }
      }
      uint32_t xw[TOK][16];
      float xb[TOK];
#pragma unroll
      for (int tt = 0; tt < TOK; ++tt) {
        const uint4* px = reinterpret_cast<const uint4*>(sx + tt * a.d + c * 32);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint4 u = px[j];
          xw[tt][4 * j] = u.x; xw[tt][4 * j + 1] = u.y;
          xw[tt][4 * j + 2] = u.z; xw[tt][4 * j + 3] = u.w;
        }
        xb[tt] = sxb[tt * C + c];
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const float s = f16_to_f32(sc[rb]);
        const uint32_t w4[4] = {q[rb].x, q[rb].y, q[rb].z, q[rb].w};
        uint32_t pr[16];
#pragma unroll
        for (int w = 0; w < 4; ++w)
#pragma unroll
          for (int k = 0; k < 4; ++k)
            pr[4 * w + k] = ((w4[w] >> (4 * k)) & 0x000F000Fu) | 0x43004300u;
#pragma unroll
        for (int tt = 0; tt < TOK; ++tt) {
          float dsum = xb[tt];
#pragma unroll
          for (int j = 0; j < 16; ++j) dsum = dot2_bf16(pr[j], xw[tt][j], dsum);
          acc[rb][tt] = fmaf(s, dsum, acc[rb][tt]);
        }
      }
    }

    // epilogue: rank-r expansions, segment reduction, store or softmax partials
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int64_t v = vbase + rb * SEG;
      const bool ok = v < a.V;
      if (ok) {
        if (a.rc) {
          float ec[TOK];
#pragma unroll
          for (int tt = 0; tt < TOK; ++tt) ec[tt] = 0.f;
          for (int64_t k = sl; k < a.rc; k += LPR) {
            const float u = float(a.cu[v * a.rc + k]);
#pragma unroll
            for (int tt = 0; tt < TOK; ++tt) ec[tt] = fmaf(u, st[tt * R + k], ec[tt]);
          }
          const float su = f16_to_f32(a.su[v]);
#pragma unroll
          for (int tt = 0; tt < TOK; ++tt) acc[rb][tt] = fmaf(su, ec[tt], acc[rb][tt]);
        }
        if (a.rr) {
          float ew[TOK];
#pragma unroll
          for (int tt = 0; tt < TOK; ++tt) ew[tt] = 0.f;
          for (int64_t k = sl; k < a.rr; k += LPR) {
            const float u = float(a.ca[v * a.rr + k]);
#pragma unroll
            for (int tt = 0; tt < TOK; ++tt) ew[tt] = fmaf(u, st[tt * R + a.rc + k], ew[tt]);
          }
          const float sa = f16_to_f32(a.sa[v]);
#pragma unroll
          for (int tt = 0; tt < TOK; ++tt) acc[rb][tt] = fmaf(sa, ew[tt], acc[rb][tt]);
        }
      }
#pragma unroll
      for (int tt = 0; tt < TOK; ++tt) acc[rb][tt] = seg_sum<LPR>(acc[rb][tt]);
      if (ok && sl == 0) {
#pragma unroll
        for (int tt = 0; tt < TOK; ++tt) {
          const float l = acc[rb][tt];
          if constexpr (!CE) {
            const int64_t o = (a.tok0 + tt) * a.ldo + v;
            if (a.out_bf16)
              reinterpret_cast<uint16_t*>(a.out)[o] = f32_to_bf16_rne(l);
            else
              reinterpret_cast<float*>(a.out)[o] = l;
          } else {
            if (l > mx[tt]) {
              se[tt] = se[tt] * fast_exp(mx[tt] - l) + 1.f;
              mx[tt] = l;
            } else {
              se[tt] += fast_exp(l - mx[tt]);
            }
            if (v == y[tt]) a.tgt_logit[a.tok0 + tt] = l;
          }
        }
      }
    }
  }

  if constexpr (CE) {
#pragma unroll
    for (int tt = 0; tt < TOK; ++tt) {
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const float om = __shfl_xor(mx[tt], off, 64);
        const float os = __shfl_xor(se[tt], off, 64);
        lse_merge(mx[tt], se[tt], om, os);
      }
      if (lane == 0) red[wid][tt] = make_float2(mx[tt], se[tt]);
    }
    __syncthreads();
    if (threadIdx.x < TOK) {
      const int tt = threadIdx.x;
      float m = red[0][tt].x, s = red[0][tt].y;
      for (int w = 1; w < kWaves; ++w) lse_merge(m, s, red[w][tt].x, red[w][tt].y);
      a.part[(a.tok0 + tt) * a.n_part + blockIdx.x] = make_float2(m, s);
    }
  }
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
using GemvFn = void (*)(GemvArgs);

template <int TOK, bool CE>
GemvFn gemv_by_lpr(int lpr) {
  switch (lpr) {
    case 1: return k_gemv<TOK, 1, CE>;
    case 2: return k_gemv<TOK, 2, CE>;
    case 4: return k_gemv<TOK, 4, CE>;
    case 8: return k_gemv<TOK, 8, CE>;
    case 16: return k_gemv<TOK, 16, CE>;
    case 32: return k_gemv<TOK, 32, CE>;
    default: return k_gemv<TOK, 64, CE>;
  }
}

template <bool CE>
GemvFn gemv_fn(int tok, int lpr) {
  switch (tok) {
    case 1: return gemv_by_lpr<1, CE>(lpr);
    case 2: return gemv_by_lpr<2, CE>(lpr);
    case 3: return gemv_by_lpr<3, CE>(lpr);
    default: return gemv_by_lpr<4, CE>(lpr);
  }
}

size_t gemv_lds_bytes(const archead_desc& d, int tok) {
  return size_t(tok) * (size_t(d.d) * 2 + size_t(d.d / 32) * 4 + size_t(d.r_c + d.r_r) * 4);
}

int64_t gemv_rows_per_step(const archead_desc& d) {
  return int64_t(kRowsPerStep) * (64 / archead::lanes_per_row(d.d));
}

archead_status hip_fail(hipError_t e, const char* what) {
  return archead::fail(ARCHEAD_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

namespace archead {

int64_t gemv_grid(const archead_handle* h, int tok, bool ce) {
  const int slot = (ce ? 8 : 0) + tok;
  archead_handle* mh = const_cast<archead_handle*>(h);
  int cached = mh->grid_cache[slot].load(std::memory_order_relaxed);
  const int64_t steps = (h->desc.V + gemv_rows_per_step(h->desc) - 1) / gemv_rows_per_step(h->desc);
  const int64_t max_blocks = (steps + kWaves - 1) / kWaves;
  if (cached <= 0) {
    const int lpr = lanes_per_row(h->desc.d);
    GemvFn fn = ce ? gemv_fn<true>(tok, lpr) : gemv_fn<false>(tok, lpr);
    int nb = 0;
    const size_t lds = gemv_lds_bytes(h->desc, tok);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, reinterpret_cast<const void*>(fn),
                                                     kBlock, lds) != hipSuccess ||
        nb <= 0)
      nb = 1;
    cached = nb * h->n_cu;
    mh->grid_cache[slot].store(cached, std::memory_order_relaxed);
  }
  return cached < max_blocks ? cached : max_blocks;
}

static size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

WsLayout ws_layout(const archead_handle* h, int64_t M, archead_op op) {
  WsLayout w;
  if (!h || M <= 0) return w;
  const archead_desc& d = h->desc;
  size_t off = 0;
  w.t_off = off;
  off = align256(off + sizeof(float) * size_t(M) * size_t(d.r_c + d.r_r));
  w.xs_off = off;
  if (op == ARCHEAD_OP_LOGITS_CE) {
    // all CE passes share one grid (the smallest of the variants used) so
    // every token row of the partials has the same number of slots
    int64_t np = 0;
    const int64_t full = M / 4, rem = M % 4;
    if (full) np = gemv_grid(h, 4, true);
    if (rem) { const int64_t g = gemv_grid(h, int(rem), true); np = (np == 0 || g < np) ? g : np; }
    w.n_part = np;
    w.part_off = off;
    off = align256(off + 2 * sizeof(float) * size_t(M) * size_t(np));
    w.tgt_off = off;
    off = align256(off + sizeof(float) * size_t(M));
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

archead_status launch_stage1(const archead_handle* h, const void* x, int64_t M, int64_t ldx,
                             float* t, hipStream_t s) {
  const archead_desc& d = h->desc;
  const int64_t R = d.r_c + d.r_r;
  if (R == 0) return ARCHEAD_OK;
  Stage1Args a;
  a.x = static_cast<const uint16_t*>(x);
  a.ldx = ldx; a.M = M; a.d = d.d;
  a.cv = static_cast<const int8_t*>(h->ptrs.core_v);
  a.sv = static_cast<const uint16_t*>(h->ptrs.core_v_scale);
  a.gv = d.r_c ? d.g_v : d.d; a.rc = d.r_c;
  a.cb = static_cast<const int8_t*>(h->ptrs.corr_b);
  a.sb = static_cast<const uint16_t*>(h->ptrs.corr_b_scale);
  a.gb = d.r_r ? d.g_b : d.d; a.rr = d.r_r;
  a.t = t;
  const int64_t waves = R * ((M + kS1Tok - 1) / kS1Tok);
  const int64_t blocks = (waves + kWaves - 1) / kWaves;
  hipLaunchKernelGGL(k_stage1, dim3(unsigned(blocks)), dim3(kBlock), 0, s, a);
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? ARCHEAD_OK : hip_fail(e, "stage-1 launch");
}

GemvArgs gemv_args(const archead_handle* h, const void* x, int64_t ldx, const float* t) {
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
  a.t = t;
  a.V = d.V; a.d = d.d; a.g = d.g; a.rc = d.r_c; a.rr = d.r_r;
  const int64_t wr = gemv_rows_per_step(d);
  a.nsteps = (d.V + wr - 1) / wr;
  a.nit = int((d.d / 32) / lanes_per_row(d.d));
  return a;
}

// One launch per group of up to 4 tokens.  forced_grid > 0 fixes the grid
// (the CE passes, whose partials are indexed by workgroup).
archead_status launch_gemv_passes(const archead_handle* h, GemvArgs a, int64_t M, bool ce,
                                  int64_t forced_grid, hipStream_t s) {
  const int lpr = lanes_per_row(h->desc.d);
  void* ev0 = h->ev_start.load(std::memory_order_relaxed);
  void* ev1 = h->ev_stop.load(std::memory_order_relaxed);
  if (ev0) {
    hipError_t e = hipEventRecord(static_cast<hipEvent_t>(ev0), s);
    if (e != hipSuccess) return hip_fail(e, "timing event record");
  }
  for (int64_t m0 = 0; m0 < M; m0 += 4) {
    const int tok = int(M - m0 < 4 ? M - m0 : 4);
    GemvFn fn = ce ? gemv_fn<true>(tok, lpr) : gemv_fn<false>(tok, lpr);
    const int64_t grid = forced_grid > 0 ? forced_grid : gemv_grid(h, tok, ce);
    a.tok0 = m0;
    const size_t lds = gemv_lds_bytes(h->desc, tok);
    if (lds > 65536) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
      if (e != hipSuccess) return hip_fail(e, "LDS size attribute");
    }
    fn<<<dim3(unsigned(grid)), dim3(kBlock), lds, s>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "GEMV launch");
  }
  if (ev1) {
    hipError_t e = hipEventRecord(static_cast<hipEvent_t>(ev1), s);
    if (e != hipSuccess) return hip_fail(e, "timing event record");
  }
  return ARCHEAD_OK;
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
  if (d.r_c && (!ptrs->core_u || !ptrs->core_u_scale || !ptrs->core_v || !ptrs->core_v_scale))
    return fail(ARCHEAD_E_INVALID_ARG, "r_c > 0 needs core_u, core_u_scale, core_v, core_v_scale");
  if (d.r_r && (!ptrs->corr_a || !ptrs->corr_a_scale || !ptrs->corr_b || !ptrs->corr_b_scale))
    return fail(ARCHEAD_E_INVALID_ARG, "r_r > 0 needs corr_a, corr_a_scale, corr_b, corr_b_scale");
  if (!aligned(ptrs->res_codes, 16)) return fail(ARCHEAD_E_MISALIGNED, "res_codes must be 16-byte aligned");
  const void* f16s[] = {ptrs->res_scales, ptrs->core_u_scale, ptrs->core_v_scale,
                        ptrs->corr_a_scale, ptrs->corr_b_scale};
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
  archead_handle* h = new (std::nothrow) archead_handle();
  if (!h) return fail(ARCHEAD_E_INVALID_ARG, "out of host memory");
  h->desc = d;
  h->ptrs = *ptrs;
  h->device = dev;
  h->n_cu = prop.multiProcessorCount;
  h->gemv_max_m.store(kDefaultGemvMaxM);
  for (auto& c : h->grid_cache) c.store(0);
  h->ev_start.store(nullptr);
  h->ev_stop.store(nullptr);
  *out = h;
  return ARCHEAD_OK;
}

void archead_destroy(archead_handle* h) { delete h; }

size_t archead_workspace_bytes(const archead_handle* h, int64_t M, archead_op op) {
  if (!h || M <= 0) return 0;
  return ws_layout(h, M, op).total;
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
  float* t = reinterpret_cast<float*>(static_cast<char*>(ws) + w.t_off);
  st = launch_stage1(h, x, M, ldx, t, s);
  if (st != ARCHEAD_OK) return st;
  GemvArgs a = gemv_args(h, x, ldx, t);
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
  char* base = static_cast<char*>(ws);
  float* t = reinterpret_cast<float*>(base + w.t_off);
  float2* part = reinterpret_cast<float2*>(base + w.part_off);
  float* tl = reinterpret_cast<float*>(base + w.tgt_off);
  st = launch_stage1(h, x, M, ldx, t, s);
  if (st != ARCHEAD_OK) return st;
  GemvArgs a = gemv_args(h, x, ldx, t);
  a.tgt = targets;
  a.tgt64 = tgt_dtype == ARCHEAD_I64;
  a.part = part;
  a.n_part = w.n_part;
  a.tgt_logit = tl;
  const int64_t n_part = w.n_part;
  st = launch_gemv_passes(h, a, M, true, n_part, s);
  if (st != ARCHEAD_OK) return st;
  hipLaunchKernelGGL(k_ce_merge, dim3(unsigned(M)), dim3(kBlock), 0, s, part, n_part, targets,
                     int(a.tgt64), tl, h->desc.V, ce);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "CE merge launch");
  if (mean_ce) {
    hipLaunchKernelGGL(k_mean, dim3(1), dim3(kBlock), 0, s, ce, M, mean_ce);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "mean launch");
  }
  return ARCHEAD_OK;
}

}  // extern "C"
