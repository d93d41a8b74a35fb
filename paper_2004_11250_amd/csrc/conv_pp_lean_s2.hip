// Pruned 3x3 conv, lean kernel at stride 2: fp32, canonical library, pad 1,
// dilation 1 (the downsampling layers of the style-transfer and colourization
// networks, Sec. 4).  A lane's patch is (2R + 1) x (2CC + 1) inputs and the
// staged tile about four times the stride-1 one, so only tilings whose rings
// still fit LDS are built.
#include "conv_pp_lean.hpp"

namespace pp {
namespace {

// (the 4 x 4 tiling with 2 waves would spill here)
constexpr bool lean_s2_id(int id) {
  return id == 45 || id == 47 || id == 49 || id == 50 || id == 52 || id == 53 || id == 54;
}

}  // namespace

long lean_lds_bytes_s2(int id) {
  switch (id) {
#define PP_L(ID, R, CC, LW, WS, V4)                                                           \
  case ID:                                                                                    \
    return lean_s2_id(ID) && kern::LGeo<R, CC, LW, WS, (V4 != 0), false, 1, 2>::fits          \
               ? kern::LGeo<R, CC, LW, WS, (V4 != 0), false, 1, 2>::LDS_FLOATS * 4L           \
               : 0L;
    PP_LRECIPES(PP_L)
#undef PP_L
    default:
      return 0;
  }
}

hipError_t launch_lean_s2(int id, const LeanParams& p, int n, bool pw, hipStream_t st) {
  switch (id) {
#define PP_L(ID, R, CC, LW, WS, V4)                                                                    \
  case ID:                                                                                             \
    if constexpr (lean_s2_id(ID)) {                                                                    \
      if (pw) return kern::launch_lean_tiling<R, CC, LW, WS, (V4 != 0), false, true, 1, 2>(p, n, st);  \
      return kern::launch_lean_tiling<R, CC, LW, WS, (V4 != 0), false, false, 1, 2>(p, n, st);         \
    } else {                                                                                           \
      return hipErrorInvalidConfiguration;                                                             \
    }
    PP_LRECIPES(PP_L)
#undef PP_L
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace pp
