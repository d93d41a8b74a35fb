// Pruned 3x3 conv, lean kernel: fp32, canonical library, stride 1, pad 1.
#include "conv_pp_lean.hpp"

namespace pp {

hipError_t launch_lean_recipe(int id, const ConvParams& c, hipStream_t st) {
  LeanParams p;
  p.blob = c.blob;
  p.x = static_cast<const float*>(c.x);
  p.y = static_cast<float*>(c.y);
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
#define PP_L(ID, R, CC, LW, WS, V4) \
  case ID:                          \
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

long lean_lds_bytes(int id) {
  switch (id) {
#define PP_L(ID, R, CC, LW, WS, V4) \
  case ID:                          \
    return kern::LGeo<R, CC, LW, WS, (V4 != 0)>::fits ? kern::LGeo<R, CC, LW, WS, (V4 != 0)>::LDS_FLOATS * 4L : 0L;
    PP_LRECIPES(PP_L)
#undef PP_L
    default:
      return 0;
  }
}

}  // namespace pp
