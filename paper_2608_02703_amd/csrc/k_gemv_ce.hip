// Instantiations of the decode GEMV kernel with the fused softmax epilogue
// (CE and argmax partials).
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

const void* gemv_ce(int tok, int lpr, bool sc8) { return gemv_fn<true, 0>(tok, lpr, sc8); }

}  // namespace kern
}  // namespace archead
