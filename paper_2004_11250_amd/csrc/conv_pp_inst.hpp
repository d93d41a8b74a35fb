// conv_pp_inst.hpp -- recipe dispatch, included by the per-library .hip files.
#pragma once

#include "conv_pp_kernel.hpp"

namespace pp {

// non-canonical libraries get a reduced set of tilings (compile time)
constexpr bool recipe_enabled(int lib, int id) {
  return lib == kLibCanon8 || id == 0 || id == 3 || id == 6 || id == 8 || id == 12 || id == 13;
}

template <int LIB, int S, int D, class TA>
hipError_t launch_recipe(int id, const ConvParams& p, hipStream_t st) {
  switch (id) {
#define PP_X(ID, R, CC, LW, WF, WS, CPW)                                            \
  case ID:                                                                          \
    if constexpr (recipe_enabled(LIB, ID))                                          \
      return kern::launch_tiling<LIB, S, D, R, CC, LW, WF, WS, CPW, TA>(p, st);     \
    else                                                                            \
      return hipErrorInvalidConfiguration;
    PP_RECIPES(PP_X)
#undef PP_X
    default:
      return hipErrorInvalidValue;
  }
}

#define PP_INSTANTIATE(LIB, S, D)                                                                   \
  template hipError_t launch_recipe<LIB, S, D, float>(int, const ConvParams&, hipStream_t);    \
  template hipError_t launch_recipe<LIB, S, D, uint16_t>(int, const ConvParams&, hipStream_t);

}  // namespace pp
