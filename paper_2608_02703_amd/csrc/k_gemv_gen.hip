// Instantiations of the decode GEMV kernel for general factor codes (ranks
// that are not multiples of 4, ARCHEAD_I5 core-left codes): 8 and 16 lanes
// per row, the widths such heads get (other widths take the byte-wise path
// of the aligned variants).
#include "dev_gemv.cuh"
#include "kernels.h"

namespace {

using GemvFn = void (*)(GemvArgs);

template <int TOK, bool CE, bool SC8, int GEN>
GemvFn gemv_by_lpr(int lpr) {
  if constexpr (GEN > 0) {   // general factor codes: the widths of small ranks only
    switch (lpr) {
      case 8: return k_gemv<TOK, 8, CE, SC8, GEN>;
      case 16: return k_gemv<TOK, 16, CE, SC8, GEN>;
      default: return nullptr;
    }
  } else {
    switch (lpr) {
      case 1: return k_gemv<TOK, 1, CE, SC8, GEN>;
      case 2: return k_gemv<TOK, 2, CE, SC8, GEN>;
      case 4: return k_gemv<TOK, 4, CE, SC8, GEN>;
      case 8: return k_gemv<TOK, 8, CE, SC8, GEN>;
      case 16: return k_gemv<TOK, 16, CE, SC8, GEN>;
      case 32: return k_gemv<TOK, 32, CE, SC8, GEN>;
      default: return k_gemv<TOK, 64, CE, SC8, GEN>;
    }
  }
}

template <bool CE, bool SC8, int GEN>
GemvFn gemv_fn_sc(int tok, int lpr) {
  switch (tok) {
    case 1: return gemv_by_lpr<1, CE, SC8, GEN>(lpr);
    case 2: return gemv_by_lpr<2, CE, SC8, GEN>(lpr);
    case 3: return gemv_by_lpr<3, CE, SC8, GEN>(lpr);
    default: return gemv_by_lpr<4, CE, SC8, GEN>(lpr);
  }
}

// the variant for the head's residual scale format (8-bit codes or fp16)
template <bool CE, int GEN>
const void* gemv_fn(int tok, int lpr, bool sc8) {
  GemvFn fn = sc8 ? gemv_fn_sc<CE, true, GEN>(tok, lpr) : gemv_fn_sc<CE, false, GEN>(tok, lpr);
  return reinterpret_cast<const void*>(fn);
}

}  // namespace

namespace archead {
namespace kern {

const void* gemv_gen(int tok, int lpr, bool ce, bool sc8, int gen) {
  if (gen == 2) return ce ? gemv_fn<true, 2>(tok, lpr, sc8) : gemv_fn<false, 2>(tok, lpr, sc8);
  return ce ? gemv_fn<true, 1>(tok, lpr, sc8) : gemv_fn<false, 1>(tok, lpr, sc8);
}

}  // namespace kern
}  // namespace archead
