// Instantiations of the MFMA decode kernel.
#include "dev_dec.cuh"
#include "kernels.h"

#ifndef ARCHEAD_DEC_GEN
#define ARCHEAD_DEC_GEN 0   // this unit's variants: aligned int8 factor codes
#endif

namespace {

using DecFn = void (*)(DecArgs);

template <bool CE, int EK, bool SC8, int GEN>
DecFn dec_fn_ek(int gw) {
  switch (gw) {
    case 1: return k_dec<1, CE, EK, SC8, GEN>;
    case 2: return k_dec<2, CE, EK, SC8, GEN>;
    default: return k_dec<4, CE, EK, SC8, GEN>;
  }
}

template <bool CE, bool SC8, int GEN>
DecFn dec_fn_sc(int gw, int ek) {
  return ek <= 2 ? dec_fn_ek<CE, 2, SC8, GEN>(gw) : dec_fn_ek<CE, 4, SC8, GEN>(gw);
}

template <int GEN>
const void* pick(int gw, bool ce, int ek, bool sc8) {
  DecFn fn = ce ? (sc8 ? dec_fn_sc<true, true, GEN>(gw, ek) : dec_fn_sc<true, false, GEN>(gw, ek))
                : (sc8 ? dec_fn_sc<false, true, GEN>(gw, ek) : dec_fn_sc<false, false, GEN>(gw, ek));
  return reinterpret_cast<const void*>(fn);
}

}  // namespace

namespace archead {
namespace kern {

const void* dec_gen(int gw, bool ce, int ek, bool sc8, int gen);

#if ARCHEAD_DEC_GEN
const void* dec_gen(int gw, bool ce, int ek, bool sc8, int gen) {
  return gen == 2 ? pick<2>(gw, ce, ek, sc8) : pick<1>(gw, ce, ek, sc8);
}
#else
const void* dec(int gw, bool ce, int ek, bool sc8, int gen) {
  return gen ? dec_gen(gw, ce, ek, sc8, gen) : pick<0>(gw, ce, ek, sc8);
}
#endif

}  // namespace kern
}  // namespace archead
