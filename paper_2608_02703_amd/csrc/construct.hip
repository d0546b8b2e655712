// Packed-head construction on the GPU (ARCHead Algorithm 1 "ARCHead
// compression" and Algorithm 2 "Expanded packed-head construction"; Section
// 3.1 for the activation metric, Section 3.2 for QuantizeCore and the
// correction fitted in that metric).
//
// From a dense head W [V, d] and calibration hidden states H [N, d]:
//   C = H^T H / N, cbar = mean diag C, C_lambda = C + lambda cbar I
//   C_lambda = Q Lambda Q^T;  T_p = Q Lambda^p Q^T,  T_p^-1 = Q Lambda^-p Q^T
//   A_c B_c = rank-r_c truncated SVD of W (A_c = U Sigma, B_c = V^T), from
//             the top eigenvectors of W^T W
//   QuantizeCore: Q5(A_c) per row, Q8(B_c) per row, Q_SC4(W - A_c B_c) in
//             groups of g along d (the residual against the UNquantized core)
//   E = W - W_d,  W_d = deq Q5(A_c) deq Q8(B_c) + deq Q_SC4(.)
//   E T_p ~ U_r Sigma_r V_r^T by a randomized SVD (Gaussian sketch of
//             r_r + oversample columns supplied by the caller, subspace
//             iterations re-orthonormalised by QR), A_w = U_r Sigma_r,
//             B_w = V_r^T T_p^-1
//   QuantizeINT8: A_w per row, B_w in groups of g_b along d
// and the codes are written in the layouts archead_create reads (INT4
// residual in ARCHEAD_INT4_V1).  All arithmetic is fp64: dense products and
// factorizations through rocBLAS / rocSOLVER, everything else in the kernels
// below.  The quantizer: scale = fp16(absmax / qmax) rounded to nearest even
// from fp64, code = clip(rint(value / scale), -qmax, qmax), zero scale and
// codes for an all-zero group.
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>
#include <rocsolver/rocsolver.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>

#include "archead.h"
#include "internal.h"

namespace {

constexpr int kB = 256;

// fp64 -> fp16 bits, IEEE round to nearest even (finite or infinite input).
__device__ uint16_t f64_to_f16_rne(double x) {
  const uint64_t b = uint64_t(__double_as_longlong(x));
  const uint16_t sign = uint16_t((b >> 48) & 0x8000u);
  const uint64_t ab = b & 0x7fffffffffffffffull;
  if (ab >= 0x7ff0000000000000ull) return ab > 0x7ff0000000000000ull ? 0x7e00 : (sign | 0x7c00);
  if (ab == 0) return sign;
  const int e = int(ab >> 52) - 1023;
  const uint64_t m = (ab & ((uint64_t(1) << 52) - 1)) | (ab >> 52 ? (uint64_t(1) << 52) : 0);
  if (e > 15) return sign | 0x7c00;
  int shift = 42;                 // keep 11 significant bits (normal fp16)
  int ee = e + 15;                // biased fp16 exponent
  if (e < -14) {                  // fp16 subnormal: units of 2^-24
    shift = 28 - e;
    ee = 0;
    if (shift >= 64) return sign;
  }
  uint64_t q = m >> shift;
  const uint64_t rem = m & ((uint64_t(1) << shift) - 1);
  const uint64_t half = uint64_t(1) << (shift - 1);
  if (rem > half || (rem == half && (q & 1))) ++q;
  if (ee == 0) return sign | uint16_t(q);          // q == 1024 is the smallest normal
  if (q == 2048) { q = 1024; ++ee; }
  if (ee >= 31) return sign | 0x7c00;
  return sign | uint16_t(ee << 10) | uint16_t(q - 1024);
}

__device__ double f16_bits_to_f64(uint16_t h) { return double(__builtin_bit_cast(_Float16, h)); }

__global__ __launch_bounds__(kB) void k_f32_to_f64(const float* src, int64_t ld, int64_t rows,
                                                   int64_t cols, double* dst) {
  const int64_t n = rows * cols;
  for (int64_t i = blockIdx.x * int64_t(kB) + threadIdx.x; i < n; i += int64_t(gridDim.x) * kB) {
    const int64_t r = i / cols, c = i - r * cols;
    dst[i] = double(src[r * ld + c]);
  }
}

// C_lambda = C + lambda * (trace C / d) I, in place; one workgroup.
__global__ __launch_bounds__(kB) void k_damp(double* C, int64_t d, double lam) {
  __shared__ double part[kB];
  double s = 0;
  for (int64_t i = threadIdx.x; i < d; i += kB) s += C[i * d + i];
  part[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0;
    for (int i = 0; i < kB; ++i) t += part[i];
    part[0] = t;
  }
  __syncthreads();
  const double add = lam * part[0] / double(d);
  for (int64_t i = threadIdx.x; i < d; i += kB) C[i * d + i] += add;
}

// out = Q diag(lam^p): column j of the column-major eigenvector array Q
// (eigenvector j) times lam[j]^p; flags[0] = 1 if an eigenvalue is <= 0.
__global__ __launch_bounds__(kB) void k_scale_eigvecs(const double* Q, const double* lam, int64_t d,
                                                      double p, double* out, int* flags) {
  const int64_t n = d * d;
  for (int64_t i = blockIdx.x * int64_t(kB) + threadIdx.x; i < n; i += int64_t(gridDim.x) * kB) {
    const int64_t j = i / d;
    const double l = lam[j];
    if (l <= 0) flags[0] = 1;
    out[i] = Q[i] * pow(l, p);
  }
}

// The top r eigenvectors (eigenvalues ascending: columns d-1, d-2, ...) of a
// column-major d x d array, in descending order, as a column-major d x r array.
__global__ __launch_bounds__(kB) void k_top_eigvecs(const double* Q, int64_t d, int64_t r,
                                                    double* out) {
  const int64_t n = d * r;
  for (int64_t i = blockIdx.x * int64_t(kB) + threadIdx.x; i < n; i += int64_t(gridDim.x) * kB) {
    const int64_t k = i / d, e = i - k * d;
    out[i] = Q[(d - 1 - k) * d + e];
  }
}

// Symmetric quantization of a rows x cols matrix (element (r, c) at
// x[r * rs + c * cs]) in groups of G consecutive columns: codes int8
// [rows][cols] (row-major), scales fp16 [rows][cols / G], and, when deq is
// not null, code * scale written at deq[r * rs + c * cs].  One thread per
// (row, group).
__global__ __launch_bounds__(kB) void k_quant(const double* x, int64_t rs, int64_t cs,
                                              int64_t rows, int64_t cols, int64_t G, int qmax,
                                              int8_t* codes, uint16_t* scales, double* deq) {
  const int64_t ng = cols / G;
  const int64_t n = rows * ng;
  for (int64_t t = blockIdx.x * int64_t(kB) + threadIdx.x; t < n; t += int64_t(gridDim.x) * kB) {
    const int64_t r = t / ng, j = t - r * ng;
    const double* xr = x + r * rs;
    double amax = 0;
    for (int64_t c = j * G; c < (j + 1) * G; ++c) amax = fmax(amax, fabs(xr[c * cs]));
    const uint16_t s16 = f64_to_f16_rne(amax / double(qmax));
    const double s = f16_bits_to_f64(s16);
    scales[t] = s16;
    for (int64_t c = j * G; c < (j + 1) * G; ++c) {
      double q = 0;
      if (s > 0) q = fmin(fmax(rint(xr[c * cs] / s), -double(qmax)), double(qmax));
      codes[r * cols + c] = int8_t(q);
      if (deq) deq[r * rs + c * cs] = q * s;
    }
  }
}

// INT4 codes [rows][d] (int8 in [-8, 7]) -> ARCHEAD_INT4_V1 bytes [rows][d/2].
__global__ __launch_bounds__(kB) void k_pack_int4(const int8_t* codes, int64_t rows, int64_t d,
                                                  uint32_t* out) {
  const int64_t nw = rows * (d / 8);
  for (int64_t w = blockIdx.x * int64_t(kB) + threadIdx.x; w < nw; w += int64_t(gridDim.x) * kB) {
    const int8_t* c = codes + w * 8;
    uint32_t q = 0;
    for (int k = 0; k < 4; ++k) {
      q |= uint32_t(c[2 * k] + 8) << (4 * k);
      q |= uint32_t(c[2 * k + 1] + 8) << (16 + 4 * k);
    }
    out[w] = q;
  }
}

// y = a - y elementwise
__global__ __launch_bounds__(kB) void k_sub_from(const double* a, double* y, int64_t n) {
  for (int64_t i = blockIdx.x * int64_t(kB) + threadIdx.x; i < n; i += int64_t(gridDim.x) * kB)
    y[i] = a[i] - y[i];
}

// rows 0 .. r-1 of the column-major k x k array V scaled by S[row]
__global__ __launch_bounds__(kB) void k_scale_rows(double* V, int64_t k, int64_t r,
                                                   const double* S) {
  const int64_t n = r * k;
  for (int64_t i = blockIdx.x * int64_t(kB) + threadIdx.x; i < n; i += int64_t(gridDim.x) * kB) {
    const int64_t row = i % r, col = i / r;
    V[col * k + row] *= S[row];
  }
}

// column-major rows x cols -> row-major [rows][cols]
__global__ __launch_bounds__(kB) void k_transpose_out(const double* src, int64_t rows,
                                                      int64_t cols, double* dst) {
  const int64_t n = rows * cols;
  for (int64_t i = blockIdx.x * int64_t(kB) + threadIdx.x; i < n; i += int64_t(gridDim.x) * kB) {
    const int64_t r = i / cols, c = i - r * cols;
    dst[i] = src[c * rows + r];
  }
}

__global__ void k_check_info(const rocblas_int* info, int* flags, int bit) {
  if (threadIdx.x == 0 && info[0] != 0) flags[0] |= bit;
}

unsigned grid_for(int64_t n) {
  const int64_t b = (n + kB - 1) / kB;
  return unsigned(std::max<int64_t>(1, std::min<int64_t>(b, 8192)));
}

size_t a256(size_t x) { return (x + 255) & ~size_t(255); }

struct BuildWs {
  size_t w, x, codes, h, c, q, t, tinv, lam, etri, vr, acc, bt, tom, z, tau, p, y2, bts,
      s, ul, vout, eg, awc, bwt, info, flags, total;
};

BuildWs build_ws(const archead_build_desc& b) {
  BuildWs o;
  const size_t V = size_t(b.V), d = size_t(b.d), N = size_t(b.N);
  const size_t rc = size_t(b.r_c), rr = size_t(b.r_r);
  const size_t k = rr ? rr + size_t(b.oversample) : 0;
  const size_t D = sizeof(double);
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t at = off; off = a256(off + bytes); return at; };
  o.w = take(D * V * d);          // W, fp64, column-major d x V (= row-major [V][d])
  o.x = take(D * V * d);          // R, then the dequantized residual, then E
  o.codes = take(V * d);          // int8 codes of the residual before packing
  o.h = take(D * N * d);          // H, fp64
  o.c = take(D * d * d);          // C_lambda, then its eigenvectors; then W^T W
  o.q = take(D * d * d);          // eigenvectors of C_lambda
  o.t = take(D * d * d);          // T_p
  o.tinv = take(D * d * d);       // T_p^-1
  o.lam = take(D * d);
  o.etri = take(D * d);
  o.vr = take(D * d * std::max<size_t>(rc, 1));     // B_c^T: d x r_c (then its dequantized copy)
  o.acc = take(D * V * std::max<size_t>(rc, 1));    // A_c: V x r_c column-major (then deq)
  o.bt = take(D * d * std::max<size_t>(rc, 1));
  o.tom = take(D * d * std::max<size_t>(k, 1));     // T_p Omega, T_p Y
  o.z = take(D * V * std::max<size_t>(k, 1));       // sketch of E T_p: V x k column-major
  o.tau = take(D * std::max<size_t>(k, 1));
  o.p = take(D * d * std::max<size_t>(k, 1));       // E^T Z
  o.y2 = take(D * d * std::max<size_t>(k, 1));
  o.bts = take(D * d * std::max<size_t>(k, 1));     // (Q^T E T_p)^T: d x k
  o.s = take(D * std::max<size_t>(k, 1));
  o.ul = take(D * d * std::max<size_t>(k, 1));
  o.vout = take(D * std::max<size_t>(k * k, 1));
  o.eg = take(D * std::max<size_t>(k, 1));
  o.awc = take(D * V * std::max<size_t>(rr, 1));    // A_w: V x r_r column-major
  o.bwt = take(D * d * std::max<size_t>(rr, 1));    // B_w^T: d x r_r column-major
  o.info = take(sizeof(rocblas_int) * 8);
  o.flags = take(sizeof(int) * 8);
  o.total = off;
  return o;
}

archead_status check_build(const archead_build_desc* b) {
  if (!b) return archead::fail(ARCHEAD_E_INVALID_ARG, "build descriptor is NULL");
  if (b->abi_version != ARCHEAD_ABI_VERSION)
    return archead::fail(ARCHEAD_E_INVALID_ARG, "abi_version %u != %u", b->abi_version,
                         ARCHEAD_ABI_VERSION);
  if (b->V <= 0 || b->d <= 0 || b->N <= 0 || b->g <= 0)
    return archead::fail(ARCHEAD_E_INVALID_ARG, "V, d, N and g must be positive");
  if (b->d % b->g || b->g % 32 || b->d % 8)
    return archead::fail(ARCHEAD_E_INVALID_ARG, "g must divide d and be a multiple of 32");
  if (b->r_c < 0 || b->r_r < 0 || b->r_c > b->d || b->r_r > b->d || b->oversample < 0 ||
      b->power_iters < 0)
    return archead::fail(ARCHEAD_E_INVALID_ARG, "ranks, oversampling, iterations out of range");
  if (b->r_r && (b->g_b <= 0 || b->d % b->g_b || b->g_b % 32))
    return archead::fail(ARCHEAD_E_INVALID_ARG, "g_b must divide d and be a multiple of 32");
  if (b->r_r && b->r_r + b->oversample > std::min(b->V, b->d))
    return archead::fail(ARCHEAD_E_INVALID_ARG, "r_r + oversample exceeds min(V, d)");
  if (!(b->p == b->p) || !(b->lambda >= 0))
    return archead::fail(ARCHEAD_E_INVALID_ARG, "p must be a number and lambda >= 0");
  // 32-bit sizes of the dense library calls
  const int64_t lim = int64_t(1) << 31;
  if (b->V >= lim || b->d >= 65536 || b->N >= lim || b->V * b->d >= (int64_t(1) << 40))
    return archead::fail(ARCHEAD_E_UNSUPPORTED, "shape too large for the construction");
  return ARCHEAD_OK;
}

}  // namespace

using archead::fail;

extern "C" {

size_t archead_build_workspace_bytes(const archead_build_desc* b) {
  if (check_build(b) != ARCHEAD_OK) return 0;
  return build_ws(*b).total;
}

archead_status archead_build_head(const archead_build_desc* b, const float* W, int64_t ldw,
                                  const float* H, int64_t ldh, const double* omega,
                                  const archead_ptrs* out, double* a_w, double* b_w, void* ws,
                                  size_t ws_bytes, void* stream) {
  archead::clear_error();
  archead_status st = check_build(b);
  if (st != ARCHEAD_OK) return st;
  const int64_t V = b->V, d = b->d, N = b->N, rc = b->r_c, rr = b->r_r;
  const int64_t k = rr ? rr + b->oversample : 0;
  if (!W || !H || !out || !ws) return fail(ARCHEAD_E_INVALID_ARG, "W, H, out and ws are required");
  if (ldw < d || ldh < d) return fail(ARCHEAD_E_INVALID_ARG, "ldw and ldh must be >= d");
  if (rr && !omega) return fail(ARCHEAD_E_INVALID_ARG, "omega is required when r_r > 0");
  if (!out->res_codes || !out->res_scales ||
      (rc && (!out->core_u || !out->core_u_scale || !out->core_v || !out->core_v_scale)) ||
      (rr && (!out->corr_a || !out->corr_a_scale || !out->corr_b || !out->corr_b_scale)))
    return fail(ARCHEAD_E_INVALID_ARG, "an output buffer of a present component is NULL");
  if ((reinterpret_cast<uintptr_t>(out->res_codes) & 3) || (reinterpret_cast<uintptr_t>(ws) & 255))
    return fail(ARCHEAD_E_MISALIGNED, "res_codes must be 4-byte and ws 256-byte aligned");
  const BuildWs L = build_ws(*b);
  if (ws_bytes < L.total) return fail(ARCHEAD_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, L.total);

  hipStream_t s = static_cast<hipStream_t>(stream);
  char* base = static_cast<char*>(ws);
  auto P = [&](size_t off) { return reinterpret_cast<double*>(base + off); };
  double *Wc = P(L.w), *X = P(L.x), *H64 = P(L.h), *C = P(L.c), *Q = P(L.q), *T = P(L.t),
         *Tinv = P(L.tinv), *lam = P(L.lam), *etri = P(L.etri), *Vr = P(L.vr), *Acc = P(L.acc),
         *Bt = P(L.bt), *TO = P(L.tom), *Z = P(L.z), *tau = P(L.tau), *Pm = P(L.p),
         *Y2 = P(L.y2), *Bts = P(L.bts), *S = P(L.s), *Ul = P(L.ul), *Vout = P(L.vout),
         *Eg = P(L.eg), *Awc = P(L.awc), *Bwt = P(L.bwt);
  int8_t* codes = reinterpret_cast<int8_t*>(base + L.codes);
  rocblas_int* info = reinterpret_cast<rocblas_int*>(base + L.info);
  int* flags = reinterpret_cast<int*>(base + L.flags);
  if (hipMemsetAsync(flags, 0, sizeof(int) * 8, s) != hipSuccess)
    return fail(ARCHEAD_E_HIP, "flag clear failed");

  rocblas_handle hb = nullptr;
  if (rocblas_create_handle(&hb) != rocblas_status_success)
    return fail(ARCHEAD_E_HIP, "rocblas_create_handle failed");
  struct HandleGuard {   // work queued on the stream finishes before the handle goes
    rocblas_handle h;
    hipStream_t s;
    ~HandleGuard() {
      (void)hipStreamSynchronize(s);
      rocblas_destroy_handle(h);
    }
  } guard{hb, s};
  rocblas_set_stream(hb, s);
  const double one = 1.0, zero = 0.0, mone = -1.0, invN = 1.0 / double(N);
  bool ok = true;
  auto chk = [&](rocblas_status r) { ok = ok && r == rocblas_status_success; };
  auto launched = [&]() { return hipGetLastError() == hipSuccess; };
  const rocblas_operation NT = rocblas_operation_none, TT = rocblas_operation_transpose;
  const rocblas_int iV = rocblas_int(V), id = rocblas_int(d), iN = rocblas_int(N),
                    irc = rocblas_int(rc), irr = rocblas_int(rr), ik = rocblas_int(k);

  // W, H to fp64 (row-major [V][d] = column-major d x V)
  hipLaunchKernelGGL(k_f32_to_f64, dim3(grid_for(V * d)), dim3(kB), 0, s, W, ldw, V, d, Wc);
  hipLaunchKernelGGL(k_f32_to_f64, dim3(grid_for(N * d)), dim3(kB), 0, s, H, ldh, N, d, H64);
  ok = ok && launched();

  // C_lambda = H^T H / N + lambda cbar I;  eigenvectors -> T_p, T_p^-1
  chk(rocblas_dgemm(hb, NT, TT, id, id, iN, &invN, H64, id, H64, id, &zero, C, id));
  hipLaunchKernelGGL(k_damp, dim3(1), dim3(kB), 0, s, C, d, b->lambda);
  chk(rocsolver_dsyevd(hb, rocblas_evect_original, rocblas_fill_upper, id, C, id, lam, etri, info));
  hipLaunchKernelGGL(k_check_info, dim3(1), dim3(64), 0, s, info, flags, 2);
  // C now holds the eigenvectors as columns (rows of the row-major view)
  hipLaunchKernelGGL(k_scale_eigvecs, dim3(grid_for(d * d)), dim3(kB), 0, s, C, lam, d, b->p, Q, flags);
  // T = sum_j lam_j^p v_j v_j^T = C diag(lam^p) C^T in column-major terms
  chk(rocblas_dgemm(hb, NT, TT, id, id, id, &one, Q, id, C, id, &zero, T, id));
  hipLaunchKernelGGL(k_scale_eigvecs, dim3(grid_for(d * d)), dim3(kB), 0, s, C, lam, d, -b->p, Q, flags);
  chk(rocblas_dgemm(hb, NT, TT, id, id, id, &one, Q, id, C, id, &zero, Tinv, id));
  ok = ok && launched();

  // QuantizeCore
  ok = ok && hipMemcpyAsync(X, Wc, sizeof(double) * V * d, hipMemcpyDeviceToDevice, s) == hipSuccess;
  if (rc) {
    // W^T W (d x d) in C; its top r_c eigenvectors are B_c^T (d x r_c)
    chk(rocblas_dgemm(hb, NT, TT, id, id, iV, &one, Wc, id, Wc, id, &zero, C, id));
    chk(rocsolver_dsyevd(hb, rocblas_evect_original, rocblas_fill_upper, id, C, id, lam, etri, info));
    hipLaunchKernelGGL(k_check_info, dim3(1), dim3(64), 0, s, info, flags, 4);
    hipLaunchKernelGGL(k_top_eigvecs, dim3(grid_for(d * rc)), dim3(kB), 0, s, C, d, rc, Vr);
    // A_c = W B_c^T: V x r_c column-major
    chk(rocblas_dgemm(hb, TT, NT, iV, irc, id, &one, Wc, id, Vr, id, &zero, Acc, iV));
    // R = W - A_c B_c (column-major d x V: X -= B_c^T A_c^T)
    chk(rocblas_dgemm(hb, NT, TT, id, iV, irc, &mone, Vr, id, Acc, iV, &one, X, id));
    // Q5(A_c) per row (element (v, k) at v + k V), dequantized in place
    hipLaunchKernelGGL(k_quant, dim3(grid_for(V)), dim3(kB), 0, s, Acc, int64_t(1), V, V, rc, rc,
                       15, static_cast<int8_t*>(const_cast<void*>(out->core_u)),
                       static_cast<uint16_t*>(const_cast<void*>(out->core_u_scale)), Acc);
    // Q8(B_c) per row (row k, column i at Vr[i + k d])
    hipLaunchKernelGGL(k_quant, dim3(grid_for(rc)), dim3(kB), 0, s, Vr, d, int64_t(1), rc, d, d,
                       127, static_cast<int8_t*>(const_cast<void*>(out->core_v)),
                       static_cast<uint16_t*>(const_cast<void*>(out->core_v_scale)), Bt);
    ok = ok && launched();
  }
  // Q_SC4(R) in groups of g, dequantized in place
  hipLaunchKernelGGL(k_quant, dim3(grid_for(V * (d / b->g))), dim3(kB), 0, s, X, d, int64_t(1), V,
                     d, b->g, 7, codes, static_cast<uint16_t*>(const_cast<void*>(out->res_scales)),
                     X);
  hipLaunchKernelGGL(k_pack_int4, dim3(grid_for(V * d / 8)), dim3(kB), 0, s, codes, V, d,
                     static_cast<uint32_t*>(const_cast<void*>(out->res_codes)));
  // E = W - deq(res) - deq(A_c) deq(B_c)
  hipLaunchKernelGGL(k_sub_from, dim3(grid_for(V * d)), dim3(kB), 0, s, Wc, X, V * d);
  ok = ok && launched();
  if (rc) chk(rocblas_dgemm(hb, NT, TT, id, iV, irc, &mone, Bt, id, Acc, iV, &one, X, id));
  double* Ec = X;   // column-major d x V

  if (rr) {
    // randomized SVD of E T_p: Z = E (T_p Omega)
    chk(rocblas_dgemm(hb, NT, NT, id, ik, id, &one, T, id, omega, id, &zero, TO, id));
    chk(rocblas_dgemm(hb, TT, NT, iV, ik, id, &one, Ec, id, TO, id, &zero, Z, iV));
    for (int64_t it = 0; it < b->power_iters; ++it) {
      chk(rocsolver_dgeqrf(hb, iV, ik, Z, iV, tau));
      chk(rocsolver_dorgqr(hb, iV, ik, ik, Z, iV, tau));
      // Y = T_p^T E^T Z  (T_p symmetric), orthonormalised
      chk(rocblas_dgemm(hb, NT, NT, id, ik, iV, &one, Ec, id, Z, iV, &zero, Pm, id));
      chk(rocblas_dgemm(hb, NT, NT, id, ik, id, &one, T, id, Pm, id, &zero, Y2, id));
      chk(rocsolver_dgeqrf(hb, id, ik, Y2, id, tau));
      chk(rocsolver_dorgqr(hb, id, ik, ik, Y2, id, tau));
      // Z = E T_p Y
      chk(rocblas_dgemm(hb, NT, NT, id, ik, id, &one, T, id, Y2, id, &zero, TO, id));
      chk(rocblas_dgemm(hb, TT, NT, iV, ik, id, &one, Ec, id, TO, id, &zero, Z, iV));
    }
    chk(rocsolver_dgeqrf(hb, iV, ik, Z, iV, tau));
    chk(rocsolver_dorgqr(hb, iV, ik, ik, Z, iV, tau));
    // (Z^T E T_p)^T = T_p (E^T Z): d x k; its SVD Ul S Vout gives
    // Z^T E T_p = Vout^T S Ul^T
    chk(rocblas_dgemm(hb, NT, NT, id, ik, iV, &one, Ec, id, Z, iV, &zero, Pm, id));
    chk(rocblas_dgemm(hb, NT, NT, id, ik, id, &one, T, id, Pm, id, &zero, Bts, id));
    chk(rocsolver_dgesvd(hb, rocblas_svect_singular, rocblas_svect_singular, id, ik, Bts, id, S,
                         Ul, id, Vout, ik, Eg, rocblas_outofplace, info));
    hipLaunchKernelGGL(k_check_info, dim3(1), dim3(64), 0, s, info, flags, 8);
    // A_w = Z Vout^T[:, :r_r] diag(S)  (V x r_r column-major)
    hipLaunchKernelGGL(k_scale_rows, dim3(grid_for(rr * k)), dim3(kB), 0, s, Vout, k, rr, S);
    chk(rocblas_dgemm(hb, NT, TT, iV, irr, ik, &one, Z, iV, Vout, ik, &zero, Awc, iV));
    // B_w^T = T_p^-1 Ul[:, :r_r]  (d x r_r column-major = row-major [r_r][d])
    chk(rocblas_dgemm(hb, NT, NT, id, irr, id, &one, Tinv, id, Ul, id, &zero, Bwt, id));
    // QuantizeINT8: A_w per row, B_w in groups of g_b
    hipLaunchKernelGGL(k_quant, dim3(grid_for(V)), dim3(kB), 0, s, Awc, int64_t(1), V, V, rr, rr,
                       127, static_cast<int8_t*>(const_cast<void*>(out->corr_a)),
                       static_cast<uint16_t*>(const_cast<void*>(out->corr_a_scale)),
                       static_cast<double*>(nullptr));
    hipLaunchKernelGGL(k_quant, dim3(grid_for(rr * (d / b->g_b))), dim3(kB), 0, s, Bwt, d,
                       int64_t(1), rr, d, b->g_b, 127,
                       static_cast<int8_t*>(const_cast<void*>(out->corr_b)),
                       static_cast<uint16_t*>(const_cast<void*>(out->corr_b_scale)),
                       static_cast<double*>(nullptr));
    if (a_w)
      hipLaunchKernelGGL(k_transpose_out, dim3(grid_for(V * rr)), dim3(kB), 0, s, Awc, V, rr, a_w);
    if (b_w)
      ok = ok && hipMemcpyAsync(b_w, Bwt, sizeof(double) * rr * d, hipMemcpyDeviceToDevice, s) ==
                     hipSuccess;
    ok = ok && launched();
  }
  if (!ok) return fail(ARCHEAD_E_HIP, "a construction step failed to launch");
  int hflags = 0;
  if (hipMemcpyAsync(&hflags, flags, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(ARCHEAD_E_HIP, "construction failed on the device");
  if (hflags & 1) return fail(ARCHEAD_E_INVALID_ARG, "damped covariance is not positive definite");
  if (hflags & 14) return fail(ARCHEAD_E_HIP, "an eigen / singular value solver did not converge");
  return ARCHEAD_OK;
}

}  // extern "C"
