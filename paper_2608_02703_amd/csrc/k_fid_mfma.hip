// Logit fidelity of the packed head against a dense bf16 head inside the
// head's V-tile pass (Section 4, "Logit Fidelity", Table 8): the tiled
// kernel's fidelity and rank variants (64-row tiles of 4 waves) and the
// per-token merge of the fidelity pass's tile statistics.
#include "dev_mfma.cuh"
#include "kernels.h"

namespace {

// One lane per token: the tiles' statistics in tile order (fp64 rescaling
// to the row maxima), giving KL(p_dense || p_packed), the summed squared
// logit error, the dense head's first argmax and the packed logit there;
// the rank is cleared for the rank pass.
__global__ void k_fidh_merge(const FidTilePart* part, int64_t n_vt, int64_t M, float* kl,
                             float* sq, int64_t* ref_idx, float* bref, int64_t* rank) {
  const int64_t m = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (m >= M) return;
  const FidTilePart* p = part + m * n_vt;
  float ma = -INFINITY, mb = -INFINITY, bat = 0.f;
  int ia = kNoIdx;
  for (int64_t c = 0; c < n_vt; ++c) {
    if (p[c].ma > ma || (p[c].ma == ma && p[c].ia < ia)) {
      ma = p[c].ma;
      ia = p[c].ia;
      bat = p[c].bat;
    }
    mb = fmaxf(mb, p[c].mb);
  }
  double sa = 0.0, sb = 0.0, t = 0.0, s2 = 0.0;
  for (int64_t c = 0; c < n_vt; ++c) {
    // a tile's sums were taken relative to its own maxima
    const double fa = exp(double(p[c].ma) - double(ma));
    const double fb = exp(double(p[c].mb) - double(mb));
    sa += double(p[c].sa) * fa;
    t += double(p[c].t) * fa;
    sb += double(p[c].sb) * fb;
    s2 += double(p[c].sq);
  }
  // sum_v p (log p - log q) with log p = a - ma - ln sa and
  // log q = b - mb - ln sb: E_p[a - b] + (mb - ma) + ln(sb / sa)
  kl[m] = float(t / sa + (double(mb) - double(ma)) + (log(sb) - log(sa)));
  sq[m] = float(s2);
  ref_idx[m] = ia == kNoIdx ? 0 : int64_t(ia);
  bref[m] = bat;
  rank[m] = 0;
}

}  // namespace

namespace archead {
namespace kern {

const void* mfma_fid(int xe) {
  return xe == 1 ? reinterpret_cast<const void*>(k_mfma<false, 64, 4, 1>)
                 : reinterpret_cast<const void*>(k_mfma<false, 64, 4, 2>);
}
const void* fid_head_merge() { return reinterpret_cast<const void*>(k_fidh_merge); }

}  // namespace kern
}  // namespace archead
