// The tiled many-token kernel's instantiations and its prologue kernels
// (head-derived tables, stage 1 on MFMA and its split-d sum).
#include "dev_mfma.cuh"
#include "kernels.h"

namespace {

__global__ __launch_bounds__(kBlock) void k_prep(PrepArgs a) {
  const int64_t nthr = int64_t(gridDim.x) * kBlock;
  const int64_t t0 = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  // (a) one thread per (vocabulary tile, column): walk the slots of the row
  // (lanes write consecutive columns)
  for (int64_t e = t0; e < a.n_vt * kTN; e += nthr) {
    const int64_t vt = e / kTN, c = e % kTN;
    const int64_t v = vt * kTN + c < a.V ? vt * kTN + c : a.V - 1;
    const uint16_t* src = a.rs + v * a.ngrp;
    const uint8_t* src8 = reinterpret_cast<const uint8_t*>(a.rs) + v * a.ngrp;
    const float rsv = a.rrs ? f16_to_f32(a.rrs[v]) : 0.f;
    float* dst = a.ratio + vt * int64_t(a.nslot) * kTN + c;
    float prev = 0.f;
    int k = 0;
    for (; k < a.ngrp; ++k) {
      float s;
      if (a.rrs) {   // rs * q, exact in fp32
        s = rsv * float(src8[k]);
        s = s == 0.f ? kZeroScale : s;
      } else {
        s = nz_scale(src[k]);
      }
      dst[int64_t(k) * kTN] = k ? prev / s : 0.f;
      prev = s;
    }
    if (a.rc) {
      const float s = nz_scale(a.su[v]);
      dst[int64_t(k++) * kTN] = prev / s;
      prev = s;
    }
    if (a.rr) {
      const float s = nz_scale(a.sa[v]);
      dst[int64_t(k++) * kTN] = prev / s;
      prev = s;
    }
    a.fin[vt * kTN + c] = prev;
  }
  // (b) 8 codes per thread
  const int64_t n8 = int64_t(a.rc + a.rr) * a.d / 8;
  for (int64_t e = t0; e < n8; e += nthr) {
    const int64_t k = e * 8 / a.d, i = e * 8 % a.d;
    const int8_t* src = k < a.rc ? a.cv + k * a.d + i : a.cb + (k - a.rc) * a.d + i;
    const uint2 w = *reinterpret_cast<const uint2*>(src);
    uint32_t o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t wj = j < 2 ? w.x : w.y;
      const int sh = 16 * (j & 1);
      const float lo = float(int8_t(wj >> sh)), hi = float(int8_t(wj >> (sh + 8)));
      o[j] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xffff0000u);
    }
    *reinterpret_cast<uint4*>(a.wbf + e * 8) = make_uint4(o[0], o[1], o[2], o[3]);
  }
  // (c) 16 bytes per thread (row-major, so lanes write consecutive chunks)
  const int64_t n16 = a.V * (a.urow / 16);
  for (int64_t e = t0; e < n16; e += nthr) {
    const int64_t v = e / (a.urow / 16);
    const int j0 = int(e % (a.urow / 16)) * 16;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int jj = 0; jj < 16; ++jj) {
      const int j = (j0 / 32) * 16 + jj;   // dimension (both copies of a block)
      int8_t c = 0;
      if (j < a.rc_pad) {
        if (j < a.rc)
          c = int8_t(fcode1(reinterpret_cast<const uint8_t*>(a.cu) + v * a.cu_row, j, a.u5 != 0));
      } else if (j - a.rc_pad < a.rr) {
        c = a.ca[v * a.rr + (j - a.rc_pad)];
      }
      w[jj / 4] |= uint32_t(uint8_t(c)) << (8 * (jj % 4));
    }
    *reinterpret_cast<uint4*>(a.ucodes + v * a.urow + j0) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

__global__ __launch_bounds__(kS1MBlock) void k_stage1m(Stage1MArgs a) {
  __shared__ float red[kS1MWaves][kS1MTok][kS1MCols + 1];
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lr = lane & 15, q = lane >> 4;
  const int R = a.rc + a.rr;
  const int64_t tok0 = int64_t(blockIdx.x) * kS1MTok;
  const int kb = blockIdx.y * kS1MCols;           // first factor row of this workgroup
  const int ngrp = a.d / a.g, cpg = a.g / 32;
  // this workgroup's residual groups (split blockIdx.z of ksplit equal
  // parts), dealt to its waves
  const int ks = blockIdx.z, gps = ngrp / a.ksplit, g0 = ks * gps;
  const int c0 = (g0 + wid * gps / kS1MWaves) * cpg, c1 = (g0 + (wid + 1) * gps / kS1MWaves) * cpg;
  const int64_t mrow = tok0 + lr < a.M ? tok0 + lr : a.M - 1;
  const uint16_t* xrow = a.x + mrow * a.ldx + 8 * q;
  const bool do_bias = blockIdx.y == 0;
  constexpr int NB = kS1MCols / 16;
  const int nblk = R - kb >= kS1MCols ? NB : (R - kb + 15) / 16;

  // this lane's factor row in each 16-column block (clamped; masked on store)
  const uint16_t* wrow[NB];
  const uint16_t* srow[NB];
  int sgrp[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    int k = kb + 16 * nb + lr;
    k = k < R ? k : (R > 0 ? R - 1 : 0);
    wrow[nb] = a.wbf + int64_t(k) * a.d + 8 * q;
    const bool core = k < a.rc;
    sgrp[nb] = core ? a.gv : a.gb;
    srow[nb] = core ? a.sv + int64_t(k) * (a.d / a.gv) : a.sb + int64_t(k - a.rc) * (a.d / a.gb);
  }
  const bf16x8_t ones = {(__bf16)1.f, (__bf16)1.f, (__bf16)1.f, (__bf16)1.f,
                         (__bf16)1.f, (__bf16)1.f, (__bf16)1.f, (__bf16)1.f};
  f32x4_t acc[NB], gs = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  bf16x8_t A, An, B[NB], Bn[NB];
  float s[NB], sn[NB];
  auto load = [&](int c, bf16x8_t& A_, bf16x8_t* B_, float* s_) {
    const int k0 = 32 * c;
    A_ = *reinterpret_cast<const bf16x8_t*>(xrow + k0);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      if (nb < nblk) {
        B_[nb] = *reinterpret_cast<const bf16x8_t*>(wrow[nb] + k0);
        s_[nb] = f16_to_f32(srow[nb][k0 / sgrp[nb]]);
      }
    }
  };
  if (c0 < c1) load(c0, A, B, s);
  for (int c = c0; c < c1; ++c) {
    if (c + 1 < c1) load(c + 1, An, Bn, sn);
    if (do_bias) gs = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, ones, gs, 0, 0, 0);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      if (nb < nblk) {
        const f32x4_t z = {0.f, 0.f, 0.f, 0.f};
        acc[nb] += s[nb] * __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B[nb], z, 0, 0, 0);
      }
    }
    if (do_bias && (c + 1) % cpg == 0) {
      const int j = c / cpg;
      if (lr == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t m = tok0 + 4 * q + i;
          if (m < a.M)
            a.gbias[((m / kTM) * a.nslot + j) * kTM + m % kTM] = -float(archead::kInt4Bias) * gs[i];
        }
      }
      gs = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    A = An;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) B[nb] = Bn[nb], s[nb] = sn[nb];
  }
  if (do_bias && ks == 0) {
    // zero biases of the expansion slots and zero padding of the split t
    const int nz = a.nslot - ngrp;
    for (int e = threadIdx.x; e < kS1MTok * nz; e += kS1MBlock) {
      const int64_t m = tok0 + e / nz;
      if (m < a.M) a.gbias[((m / kTM) * a.nslot + ngrp + e % nz) * kTM + m % kTM] = 0.f;
    }
    const int pu = kExpDims * a.nch_u;   // padded dimensions of the U_c part
    for (int e = threadIdx.x; e < kS1MTok * a.nch * 64; e += kS1MBlock) {
      const int tt = e / (a.nch * 64), j = e % (a.nch * 64), blk = j / 64, w = j % 64;
      const int dim = blk * kExpDims + w % kExpDims;
      const bool pad = w >= 48 || (dim < pu ? dim >= a.rc : dim - pu >= a.rr);
      const int64_t m = tok0 + tt;
      if (m < a.M && pad) a.tsplit[(m * a.nch + blk) * 64 + w] = 0;
    }
  }
  if (R == 0) return;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wid][4 * q + i][16 * nb + lr] = acc[nb][i];
  __syncthreads();
  for (int e = threadIdx.x; e < kS1MTok * kS1MCols; e += kS1MBlock) {
    const int tt = e / kS1MCols, c = e % kS1MCols;
    const int64_t m = tok0 + tt;
    const int k = kb + c;
    if (m < a.M && k < R) {
      float v = red[0][tt][c];
#pragma unroll
      for (int w = 1; w < kS1MWaves; ++w) v += red[w][tt][c];
      if (a.ksplit > 1) {
        a.tpart[(int64_t(ks) * a.M + m) * R + k] = v;
        continue;
      }
      const __bf16 hi = (__bf16)v;
      const float r1 = v - float(hi);
      const __bf16 md = (__bf16)r1;
      const __bf16 lo = (__bf16)(r1 - float(md));
      const int dim = k < a.rc ? k : kExpDims * a.nch_u + (k - a.rc);
      uint16_t* dst = a.tsplit + (m * a.nch + dim / kExpDims) * 64 + dim % kExpDims;
      dst[0] = __builtin_bit_cast(uint16_t, hi);
      dst[16] = __builtin_bit_cast(uint16_t, md);
      dst[32] = __builtin_bit_cast(uint16_t, lo);
    }
  }
}

// t[m][k] as the sum of the ksplit partials in split order, then split
// into three bf16 parts as k_stage1m does when it is not split.
__global__ __launch_bounds__(kBlock) void k_stage1m_fin(Stage1MArgs a) {
  const int R = a.rc + a.rr;
  const int64_t e = int64_t(blockIdx.x) * kBlock + threadIdx.x;
  if (e >= a.M * R) return;
  const int64_t m = e / R;
  const int k = int(e % R);
  float v = a.tpart[m * R + k];
  for (int ks = 1; ks < a.ksplit; ++ks) v += a.tpart[(int64_t(ks) * a.M + m) * R + k];
  const __bf16 hi = (__bf16)v;
  const float r1 = v - float(hi);
  const __bf16 md = (__bf16)r1;
  const __bf16 lo = (__bf16)(r1 - float(md));
  const int dim = k < a.rc ? k : kExpDims * a.nch_u + (k - a.rc);
  uint16_t* dst = a.tsplit + (m * a.nch + dim / kExpDims) * 64 + dim % kExpDims;
  dst[0] = __builtin_bit_cast(uint16_t, hi);
  dst[16] = __builtin_bit_cast(uint16_t, md);
  dst[32] = __builtin_bit_cast(uint16_t, lo);
}


}  // namespace

namespace archead {
namespace kern {

const void* mfma(bool ce, int tm, int nw) {
  if (tm == 64 && nw == 4)
    return ce ? reinterpret_cast<const void*>(k_mfma<true, 64, 4>)
              : reinterpret_cast<const void*>(k_mfma<false, 64, 4>);
  if (tm == 128 && nw == 4)
    return ce ? reinterpret_cast<const void*>(k_mfma<true, 128, 4>)
              : reinterpret_cast<const void*>(k_mfma<false, 128, 4>);
  if (tm == 128)
    return ce ? reinterpret_cast<const void*>(k_mfma<true, 128, 8>)
              : reinterpret_cast<const void*>(k_mfma<false, 128, 8>);
  return ce ? reinterpret_cast<const void*>(k_mfma<true, kTM, 8>)
            : reinterpret_cast<const void*>(k_mfma<false, kTM, 8>);
}
const void* prep() { return reinterpret_cast<const void*>(k_prep); }
const void* stage1m() { return reinterpret_cast<const void*>(k_stage1m); }
const void* stage1m_fin() { return reinterpret_cast<const void*>(k_stage1m_fin); }

}  // namespace kern
}  // namespace archead
