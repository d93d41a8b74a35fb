// Pruned 3x3 conv, lean kernel: fp32 or bf16, canonical library, stride 1, pad 1.
#include "conv_pp_lean.hpp"

namespace pp {

// the fp32 tilings also built to read prepared weights (those the planner picks)
constexpr bool lean_pw_id(int id) {
  return id == 40 || id == 56 || id == 46 || id == 55 || id == 58 || id == 59 || id == 48 || id == 51 || id == 54;
}

// the tilings also built for bf16 activations (those the planner picks for
// bf16 layers, and their 4-byte staging twins).  The 16-wave 2 x 4 tilings
// spill a few dozen bytes per lane at bf16's register count (128 at four
// waves per SIMD), yet on 56 x 56 maps they still beat the 8-wave 2 x 4 ones
// by 5-15 %, with or without prepared weights
constexpr bool lean_bf_tiling(int id) {
  return id == 40 || id == 56 || id == 46 || id == 55 || id == 58 || id == 59 || id == 48 || id == 51 || id == 54;
}

bool lean_pw_tiling(int id) { return lean_pw_id(id); }

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
  p.wprep = static_cast<const uint8_t*>(c.wprep);
  const bool pw = c.wprep != nullptr;
  p.groups = make_fastdiv(c.n_groups);
  // (stride, dilation = pad): (1, 1); fp32 also (1, 2) and (2, 1)
  const bool ok = c.pad == c.dil && ((c.stride == 1 && c.dil == 1) ||
                                     (!bf16 && ((c.stride == 1 && c.dil == 2) || (c.stride == 2 && c.dil == 1))));
  if (!ok) return hipErrorInvalidValue;
  if (c.dil == 2) return launch_lean_d2(id, p, c.n, pw, st);
  if (c.stride == 2) return launch_lean_s2(id, p, c.n, pw, st);
  switch (id) {
#define PP_L(ID, R, CC, LW, WS, V4)                                                          \
  case ID:                                                                                   \
    if constexpr (lean_bf_tiling(ID)) {                                                      \
      if (bf16 && pw) return kern::launch_lean_tiling<R, CC, LW, WS, (V4 != 0), true, true>(p, c.n, st); \
      if (bf16) return kern::launch_lean_tiling<R, CC, LW, WS, (V4 != 0), true>(p, c.n, st); \
    } else {                                                                                 \
      if (bf16) return hipErrorInvalidConfiguration;                                         \
    }                                                                                        \
    if constexpr (lean_pw_id(ID)) {                                                          \
      if (pw) return kern::launch_lean_tiling<R, CC, LW, WS, (V4 != 0), false, true>(p, c.n, st); \
    } else {                                                                                 \
      if (pw) return hipErrorInvalidConfiguration;                                           \
    }                                                                                        \
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

long lean_lds_bytes(int id, bool bf16, int dil, int stride) {
  if (stride == 2) return bf16 || dil != 1 ? 0L : lean_lds_bytes_s2(id);
  if (dil == 2) return bf16 || stride != 1 ? 0L : lean_lds_bytes_d2(id);
  if (dil != 1 || stride != 1) return 0L;
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

// the prepared weights of a layer: entry (group, channel) holds its 8 slots'
// 4 taps (pattern tap order, as stored), zeros for pruned slots; one thread
// per float.  Every offset read from the blob is clamped to the weights it
// holds.
__global__ __launch_bounds__(256) void pp_lean_expand_kernel(const uint8_t* blob, uint32_t off_woff, uint32_t off_w,
                                                             uint32_t n_wt, uint32_t n_entries, int bf16_w,
                                                             float* out) {
  const uint32_t i = blockIdx.x * 256u + threadIdx.x;
  if (i >= n_entries * 32u) return;
  const uint32_t e = i >> 5, j = i & 31u, s = j >> 2, t = j & 3u;
  const uint32_t wo = reinterpret_cast<const uint32_t*>(blob + off_woff)[e];
  const uint32_t kept = wo >> 24;
  float v = 0.0f;
  if ((kept >> s) & 1u) {
    const uint32_t k = min((wo & 0xFFFFFFu) + 4u * __builtin_popcount(kept & ((1u << s) - 1u)) + t,
                           n_wt ? n_wt - 1 : 0u);
    // bf16 weights widen exactly
    v = bf16_w ? __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(blob + off_w)[k]) << 16)
               : reinterpret_cast<const float*>(blob + off_w)[k];
  }
  out[i] = v;
}

size_t lean_prepared_bytes(const ConvParams& p) { return static_cast<size_t>(p.n_groups) * p.c_in * 32u * sizeof(float); }

hipError_t launch_lean_expand(const ConvParams& p, bool bf16_w, void* out, hipStream_t st) {
  const size_t n = static_cast<size_t>(p.n_groups) * p.c_in;
  if (n == 0 || n * 32 > 0xFFFFFFFFull) return hipErrorInvalidValue;
  const uint32_t blocks = static_cast<uint32_t>((n * 32 + 255) / 256);
  hipLaunchKernelGGL(pp_lean_expand_kernel, dim3(blocks), dim3(256), 0, st, p.blob, p.off_woff, p.off_w, p.n_wt,
                     static_cast<uint32_t>(n), bf16_w ? 1 : 0, static_cast<float*>(out));
  return hipGetLastError();
}

}  // namespace pp
