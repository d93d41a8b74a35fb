// Pruned 3x3 conv, lean kernel at dilation 2: fp32, canonical library,
// stride 1, pad 2 (the dilated layers of the colourization network, Sec. 4).
// The same tilings as at dilation 1 (those the planner picks for fp32
// layers), with a halo of 2 and every tap offset doubled.
#include "conv_pp_lean.hpp"

namespace pp {
namespace {

// (the 16-wave 2 x 4 tilings would spill at dilation 2's larger patch)
constexpr bool lean_d2_id(int id) {
  return id == 40 || id == 56 || id == 46 || id == 55 || id == 48 || id == 51 || id == 54;
}

}  // namespace

long lean_lds_bytes_d2(int id) {
  switch (id) {
#define PP_L(ID, R, CC, LW, WS, V4)                                                           \
  case ID:                                                                                    \
    return lean_d2_id(ID) && kern::LGeo<R, CC, LW, WS, (V4 != 0), false, 2>::fits             \
               ? kern::LGeo<R, CC, LW, WS, (V4 != 0), false, 2>::LDS_FLOATS * 4L              \
               : 0L;
    PP_LRECIPES(PP_L)
#undef PP_L
    default:
      return 0;
  }
}

hipError_t launch_lean_d2(int id, const LeanParams& p, int n, bool pw, hipStream_t st) {
  switch (id) {
#define PP_L(ID, R, CC, LW, WS, V4)                                                                  \
  case ID:                                                                                           \
    if constexpr (lean_d2_id(ID)) {                                                                  \
      if (pw) return kern::launch_lean_tiling<R, CC, LW, WS, (V4 != 0), false, true, 2>(p, n, st);  \
      return kern::launch_lean_tiling<R, CC, LW, WS, (V4 != 0), false, false, 2>(p, n, st);         \
    } else {                                                                                         \
      return hipErrorInvalidConfiguration;                                                           \
    }
    PP_LRECIPES(PP_L)
#undef PP_L
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace pp
