// Pruned 3x3 conv, lean kernel: fp32 or bf16, canonical library, stride 1, pad 1.
#include "conv_pp_lean.hpp"

namespace pp {

// the tilings also built for bf16 activations (those the planner picks for
// bf16 layers, and their 4-byte staging twins; the 16-wave 2 x 4 tilings
// would spill at bf16's register count)
constexpr bool lean_bf_tiling(int id) {
  return id == 40 || id == 56 || id == 46 || id == 55 || id == 48 || id == 51 || id == 54;
}

hipError_t launch_lean_recipe(int id, const ConvParams& c, bool bf16, hipStream_t st) {
  LeanParams p;
  p.blob = c.blob;
  p.x = c.x;
  p.y = c.y;
  p.part = c.part;
  p.h = c.h;
  p.w = c.w;
  p.ho = c.ho;
  p.wo = c.wo;
  p.c_in = c.c_in;
  p.c_out = c.c_out;
  p.off_codes = c.off_codes;
  p.off_woff = c.off_woff;
  p.off_w = c.off_w;
  p.off_bias = c.off_bias;
  p.off_perm = c.off_perm;
  p.blob_bytes = c.blob_bytes;
  p.flags = c.flags;
  p.ksplit = c.ksplit;
  p.groups = make_fastdiv(c.n_groups);
  switch (id) {
#define PP_L(ID, R, CC, LW, WS, V4)                                                   \
  case ID:                                                                            \
    if constexpr (lean_bf_tiling(ID)) {                                               \
      if (bf16) return kern::launch_lean_tiling<R, CC, LW, WS, (V4 != 0), true>(p, c.n, st); \
    } else {                                                                          \
      if (bf16) return hipErrorInvalidConfiguration;                                  \
    }                                                                                 \
    return kern::launch_lean_tiling<R, CC, LW, WS, (V4 != 0)>(p, c.n, st);
    PP_LRECIPES(PP_L)
#undef PP_L
    default:
      return hipErrorInvalidValue;
  }
}

bool lean_v4(int id) {
  switch (id) {
#define PP_L(ID, R, CC, LW, WS, V4) \
  case ID:                          \
    return V4 != 0;
    PP_LRECIPES(PP_L)
#undef PP_L
    default:
      return false;
  }
}

long lean_lds_bytes(int id, bool bf16) {
  switch (id) {
#define PP_L(ID, R, CC, LW, WS, V4)                                                                     \
  case ID:                                                                                              \
    if (bf16)                                                                                           \
      return lean_bf_tiling(ID) && kern::LGeo<R, CC, LW, WS, (V4 != 0), true>::fits                     \
                 ? kern::LGeo<R, CC, LW, WS, (V4 != 0), true>::LDS_FLOATS * 4L                          \
                 : 0L;                                                                                  \
    return kern::LGeo<R, CC, LW, WS, (V4 != 0)>::fits ? kern::LGeo<R, CC, LW, WS, (V4 != 0)>::LDS_FLOATS * 4L : 0L;
    PP_LRECIPES(PP_L)
#undef PP_L
    default:
      return 0;
  }
}

}  // namespace pp
