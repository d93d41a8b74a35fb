// conv_pp_wave_inst.hpp -- dispatch over the wave-pipeline tilings, included
// by the per-(stride, dilation) .hip files.
#pragma once

#include "conv_pp_wave.hpp"

namespace pp {

// the register-pipelined tilings exist for fp32 and the canonical library
template <int LIB, int S, int D, class TA>
hipError_t launch_wave_recipe(int id, const ConvParams& p, hipStream_t st) {
  constexpr bool kPipeOk = LIB == kLibCanon8 && sizeof(TA) == 4;
  switch (id) {
#define PP_W(ID, R, CC, LW, WS, P)                                                    \
  case ID:                                                                            \
    if constexpr (!P || kPipeOk)                                                      \
      return kern::launch_wave_tiling<LIB, S, D, R, CC, LW, WS, (P != 0), TA>(p, st); \
    else                                                                              \
      return hipErrorInvalidValue;
    PP_WRECIPES(PP_W)
#undef PP_W
    default:
      return hipErrorInvalidValue;
  }
}

#define PP_WAVE_INSTANTIATE(LIB, S, D)                                                         \
  template hipError_t launch_wave_recipe<LIB, S, D, float>(int, const ConvParams&, hipStream_t); \
  template hipError_t launch_wave_recipe<LIB, S, D, uint16_t>(int, const ConvParams&, hipStream_t);

}  // namespace pp
