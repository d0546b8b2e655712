// Instantiations of the several-token kernel.
#include "dev_mid.cuh"
#include "kernels.h"

#ifndef ARCHEAD_MID_GEN
#define ARCHEAD_MID_GEN 0   // this unit's variants: aligned int8 factor codes
#endif

namespace {

using MidFn = void (*)(MidArgs);

// Tiles of 32 tokens (two MFMA row blocks) and 3 units per wave, for both
// group sizes (the main loop walks 128 codes per step either way).  (Tiles
// of 64 tokens with 2 units per wave measured slower than two tiles of 32.)
template <bool CE, int GEN>
MidFn mid_fn(int gw, bool sc8) {
  if (sc8) return gw == 4 ? k_mid<4, 2, 3, CE, true, GEN> : k_mid<2, 2, 3, CE, true, GEN>;
  return gw == 4 ? k_mid<4, 2, 3, CE, false, GEN> : k_mid<2, 2, 3, CE, false, GEN>;
}

template <int GEN>
const void* pick(int gw, bool ce, bool sc8) {
  MidFn fn = ce ? mid_fn<true, GEN>(gw, sc8) : mid_fn<false, GEN>(gw, sc8);
  return reinterpret_cast<const void*>(fn);
}

}  // namespace

namespace archead {
namespace kern {

const void* mid_gen(int gw, bool ce, bool sc8, int gen);

#if ARCHEAD_MID_GEN
const void* mid_gen(int gw, bool ce, bool sc8, int gen) {
  return gen == 2 ? pick<2>(gw, ce, sc8) : pick<1>(gw, ce, sc8);
}
#else
const void* mid(int gw, bool ce, bool sc8, int gen) {
  return gen ? mid_gen(gw, ce, sc8, gen) : pick<0>(gw, ce, sc8);
}
#endif

}  // namespace kern
}  // namespace archead
