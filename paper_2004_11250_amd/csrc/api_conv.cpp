// api_conv.cpp -- pp_conv2d_fwd / pp_conv2d_out_size: host validation and
// dispatch of the pruned 3x3 convolution (pattern + connectivity pruning,
// Sec. 2; conv fused with bias and activation, Sec. 3).
#include <hip/hip_runtime.h>

#include <cstring>
#include <string>

#include "api_internal.hpp"
#include "conv_pp.hpp"
#include "ppk1.hpp"

namespace pp {

static const uint16_t kCanon8Masks[8] = {0x03A, 0x0B2, 0x0B8, 0x09A, 0x01B, 0x036, 0x0D8, 0x1B0};

int library_kind(const BlobView& v) {
  if (v.n_patterns == 8) {
    bool same = true;
    for (int p = 0; p < 8; ++p) {
      uint16_t m;
      std::memcpy(&m, v.masks + p, 2);
      same = same && m == kCanon8Masks[p];
    }
    if (same) return kLibCanon8;
  }
  if (v.n_patterns == 1) {
    uint16_t m;
    std::memcpy(&m, v.masks, 2);
    if (m == 0x1FF) return kLibDense9;
  }
  return kLibGeneric;
}

static int out_dim(int in, int pad, int dil, int stride) { return (in + 2 * pad - 2 * dil - 1) / stride + 1; }

pp_status conv_check(const BlobView& v, int32_t n, int32_t h, int32_t w, int32_t act_dtype, int* ho, int* wo) {
  if (n < 1 || h < 1 || w < 1) return fail(PP_EINVAL, "n, h, w must be >= 1");
  if (act_dtype != PP_F32 && act_dtype != PP_BF16) return fail(PP_EINVAL, "bad activation dtype");
  if (v.stride != 1 && v.stride != 2) return fail(PP_EUNSUPPORTED, "stride must be 1 or 2");
  if (v.dil != 1 && v.dil != 2) return fail(PP_EUNSUPPORTED, "dilation must be 1 or 2");
  if (v.pad > 2 * v.dil) return fail(PP_EUNSUPPORTED, "pad larger than the kernel extent");
  if (v.wdtype != act_dtype) return fail(PP_EUNSUPPORTED, "weight dtype must equal activation dtype");
  const long hn = h + 2L * v.pad - 2L * v.dil - 1, wn = w + 2L * v.pad - 2L * v.dil - 1;
  if (hn < 0 || wn < 0) return fail(PP_EUNSUPPORTED, "input smaller than the dilated kernel");
  if (static_cast<long long>(n) * v.c_in * h * w > (1LL << 40) ||
      static_cast<long long>(n) * v.c_out * h * w > (1LL << 40))
    return fail(PP_EINVAL, "tensor too large");
  // the kernels address one image of x through a buffer resource with byte
  // offsets below 2^31
  const long long esz = act_dtype == PP_BF16 ? 2 : 4;
  if (static_cast<long long>(v.c_in) * h * w * esz >= (1LL << 31))
    return fail(PP_EUNSUPPORTED, "one input image must be smaller than 2 GiB");
  *ho = out_dim(h, v.pad, v.dil, v.stride);
  *wo = out_dim(w, v.pad, v.dil, v.stride);
  return PP_OK;
}

ConvParams layer_params(const BlobView& v, int32_t n, int32_t h, int32_t w, int ho, int wo);

ConvPlan plan_with_scratch(const ConvParams& p, int kind, bool bf16, size_t scratch_bytes, bool no_lean) {
  ConvPlan pl = plan_conv(p, kind, bf16, scratch_bytes > 0, no_lean);
  if (split_bytes(pl, p) > scratch_bytes) pl = plan_conv(p, kind, bf16, false, no_lean);   // no room: no split
  return pl;
}

int conv_recipe(const BlobView& v, int32_t n, int32_t h, int32_t w, int32_t act_dtype, uint32_t flags,
                size_t scratch_bytes) {
  const bool up = (flags & PP_UPSAMPLE2) != 0;
  int ho = 0, wo = 0;
  if (conv_check(v, n, up ? 2 * h : h, up ? 2 * w : w, act_dtype, &ho, &wo) != PP_OK) return -1;
  ConvParams p = layer_params(v, n, up ? 2 * h : h, up ? 2 * w : w, ho, wo);
  p.flags = flags;
  return plan_with_scratch(p, library_kind(v), act_dtype == PP_BF16, scratch_bytes, false).recipe;
}

static size_t align256(size_t n) { return (n + 255) / 256 * 256; }

pp_status conv_enqueue(const BlobView& v, const void* d_blob, const void* x, void* y, int32_t n, int32_t h,
                       int32_t w, int32_t act_dtype, uint32_t flags, void* scratch, size_t scratch_bytes,
                       hipStream_t st, const void* wprep) {
  // with PP_UPSAMPLE2 the conv's input is x upsampled to 2h x 2w
  const bool up = (flags & PP_UPSAMPLE2) != 0;
  if (up && (h < 1 || w < 1 || h > (1 << 29) || w > (1 << 29))) return fail(PP_EINVAL, "bad h, w");
  const int hv = up ? 2 * h : h, wv = up ? 2 * w : w;
  int ho = 0, wo = 0;
  pp_status s = conv_check(v, n, hv, wv, act_dtype, &ho, &wo);
  if (s != PP_OK) return s;
  if (!d_blob || !x || !y) return fail(PP_EINVAL, "NULL device pointer");
  if (reinterpret_cast<uintptr_t>(d_blob) % 256) return fail(PP_EINVAL, "device blob must be 256-byte aligned");
  const size_t esz = act_dtype == PP_BF16 ? 2 : 4;
  if (reinterpret_cast<uintptr_t>(x) % esz || reinterpret_cast<uintptr_t>(y) % esz)
    return fail(PP_EINVAL, "activation pointers misaligned");
  if (flags & ~static_cast<uint32_t>(PP_RELU | PP_MAXPOOL2 | PP_ACCUMULATE | PP_PIXSHUF2 | PP_UPSAMPLE2 | PP_PREPARED))
    return fail(PP_EINVAL, "unknown flags");
  // PP_PREPARED: the workspace starts with the layer's prepared weights (the
  // matrix-core form's and / or the lean kernel's), read only by the plans
  // they are for
  const bool prepared = (flags & PP_PREPARED) != 0;
  flags &= ~static_cast<uint32_t>(PP_PREPARED);
  if (prepared && (!scratch || reinterpret_cast<uintptr_t>(scratch) % 256))
    return fail(PP_EINVAL, "PP_PREPARED needs the prepared weights (256-byte aligned) as the workspace");
  if (prepared && scratch_bytes < prepared_bytes(v))
    return fail(PP_ESIZE, "prepared weights smaller than pp_conv2d_prepare writes");
  if (wprep && reinterpret_cast<uintptr_t>(wprep) % 256) return fail(PP_EINVAL, "prepared weights misaligned");
  {
    const uint32_t f = flags & (PP_MAXPOOL2 | PP_ACCUMULATE | PP_PIXSHUF2);
    if (f & (f - 1)) return fail(PP_EINVAL, "more than one of PP_MAXPOOL2, PP_ACCUMULATE, PP_PIXSHUF2");
  }
  if ((flags & PP_PIXSHUF2) && v.c_out % 4) return fail(PP_EINVAL, "PP_PIXSHUF2 needs c_out a multiple of 4");
  const bool pool = (flags & PP_MAXPOOL2) != 0;
  if (pool && (ho < 2 || wo < 2)) return fail(PP_EINVAL, "pooled output needs h_out, w_out >= 2");
  const uint8_t* xb = static_cast<const uint8_t*>(x);
  const uint8_t* yb = static_cast<const uint8_t*>(y);
  const size_t xbytes = static_cast<size_t>(n) * v.c_in * h * w * esz;
  const size_t ybytes = static_cast<size_t>(n) * v.c_out * (pool ? (ho / 2) * (wo / 2) : ho * wo) * esz;
  if (xb < yb + ybytes && yb < xb + xbytes) return fail(PP_EINVAL, "x and y overlap");

  ConvParams p = layer_params(v, n, hv, wv, ho, wo);
  p.blob = static_cast<const uint8_t*>(d_blob);
  p.x = x;
  p.y = y;
  p.flags = flags;
  const int lib = library_kind(v);
  const bool bf = act_dtype == PP_BF16;
  if (prepared) {
    // the workspace starts with the prepared weights; bytes past them
    // (from the next 256-byte boundary) serve as split scratch
    void* const pw = scratch;
    const size_t head = align256(prepared_bytes(v));
    void* const tail = scratch_bytes > head ? static_cast<uint8_t*>(scratch) + head : nullptr;
    const size_t tail_bytes = tail ? scratch_bytes - head : 0;
    wprep = lean_prepared(v, pw);   // the lean kernel's weights (when it runs)
    if (bf) {
      // the matrix-core form's weights; any other plan ignores them
      ConvParams q = p;
      const ConvPlan mp = plan_with_scratch(q, lib, bf, scratch_bytes, false);
      if (mp.recipe == kRecipeMfma) {
        q.part = static_cast<float*>(pw);
        q.flags |= PP_PREPARED;   // the expansion is skipped
        const hipError_t e = launch_conv(lib, mp, q, bf, st);
        if (e != hipSuccess) return fail(PP_EHIP, std::string("conv launch: ") + hipGetErrorString(e));
        return PP_OK;
      }
    }
    scratch = tail;
    scratch_bytes = tail_bytes;
  }
  const size_t usable = reinterpret_cast<uintptr_t>(scratch) % 256 ? 0 : scratch_bytes;
  // the plan for library kind `kind`; a split only with enough scratch
  auto make_plan = [&](int kind, ConvParams* pp_, bool no_lean) {
    ConvPlan pl = plan_with_scratch(*pp_, kind, bf, scratch != nullptr ? usable : 0, no_lean);
    if (split_bytes(pl, *pp_) > 0) pp_->part = static_cast<float*>(scratch);
    return pl;
  };
  if (lib == kLibGeneric && jit_library4(v)) {
    // a 4-tap library with run-time compiled kernels (pp_jit_library): as
    // the canonical library's plan
    ConvParams jp = p;
    const ConvPlan pl = make_plan(kLibCanon8, &jp, true);
    hipError_t e = hipSuccess;
    if (pl.recipe >= kFirstWaveRecipe && pl.recipe < kNumRecipes && jit_launch(v, pl, jp, bf, st, &e)) {
      if (e != hipSuccess) return fail(PP_EHIP, std::string("conv launch: ") + hipGetErrorString(e));
      return PP_OK;
    }
  }
  ConvPlan plan = make_plan(lib, &p, false);
  if (plan.recipe < 0) return fail(PP_EUNSUPPORTED, "no tiling fuses the upsampling / max pool / accumulation / pixel shuffle for this layer");
  // prepared lean weights: read by the lean tilings built for them, ignored by any other plan
  if (wprep && is_lean_recipe(plan.recipe) && lean_pw_tiling(plan.recipe)) p.wprep = wprep;
  hipError_t e = launch_conv(lib, plan, p, bf, st);
  if (e != hipSuccess) return fail(PP_EHIP, std::string("conv launch: ") + hipGetErrorString(e));
  return PP_OK;
}

bool conv_fusable(const BlobView& v, int32_t n, int32_t h, int32_t w, int32_t act_dtype, uint32_t flags,
                  bool with_scratch) {
  int ho = 0, wo = 0;
  if (conv_check(v, n, h, w, act_dtype, &ho, &wo) != PP_OK) return false;
  if ((flags & PP_MAXPOOL2) && (ho < 2 || wo < 2)) return false;
  if ((flags & PP_PIXSHUF2) && v.c_out % 4) return false;
  if ((flags & PP_UPSAMPLE2) && (h % 2 || w % 2)) return false;
  ConvParams p = layer_params(v, n, h, w, ho, wo);
  p.flags = flags;
  const int lib = library_kind(v);
  const bool bf = act_dtype == PP_BF16;
  if (plan_conv(p, lib, bf, with_scratch).recipe < 0) return false;
  // a bf16 conv that runs on the lean kernel unfused is not fused with an
  // upsample or a pixel shuffle, which that kernel does not take: the fused
  // conv would run on another kernel, whose sums round differently
  if (bf && (flags & (PP_UPSAMPLE2 | PP_PIXSHUF2))) {
    ConvParams q = p;
    q.flags = flags & ~static_cast<uint32_t>(PP_UPSAMPLE2 | PP_PIXSHUF2);
    if (is_lean_recipe(plan_conv(q, lib, bf, with_scratch).recipe)) return false;
  }
  return true;
}

size_t conv_scratch_bytes(const BlobView& v, int32_t n, int32_t h, int32_t w, int32_t act_dtype) {
  int ho = 0, wo = 0;
  if (conv_check(v, n, h, w, act_dtype, &ho, &wo) != PP_OK) return 0;
  const ConvParams p = layer_params(v, n, h, w, ho, wo);
  return split_bytes(plan_conv(p, library_kind(v), act_dtype == PP_BF16, true), p);
}

// launch parameters of one layer for an n x c_in x h x w input (device
// pointers and flags are set by the caller)
ConvParams layer_params(const BlobView& v, int32_t n, int32_t h, int32_t w, int ho, int wo) {
  ConvParams p;
  p.n = n;
  p.h = h;
  p.w = w;
  p.ho = ho;
  p.wo = wo;
  p.c_in = v.c_in;
  p.c_out = v.c_out;
  p.pad = v.pad;
  p.stride = v.stride;
  p.dil = v.dil;
  p.n_groups = v.n_groups;
  p.off_codes = v.off_codes;
  p.off_woff = v.off_woff;
  p.off_w = v.off_w;
  p.off_bias = v.off_bias;
  p.off_perm = v.off_perm;
  p.off_masks = v.off_masks;
  p.n_wt = static_cast<uint32_t>(v.n_wt);
  p.blob_bytes = static_cast<uint32_t>(v.total);
  p.n_patterns = v.n_patterns;
  return p;
}

}  // namespace pp

using namespace pp;

extern "C" pp_status pp_conv2d_out_size(const void* h_blob, size_t blob_bytes, int32_t h, int32_t w,
                                        int32_t* h_out, int32_t* w_out) {
  clear_error();
  BlobView v;
  pp_status s = parse_blob(h_blob, blob_bytes, &v, /*full=*/false);
  if (s != PP_OK) return s;
  if (h < 1 || w < 1) return fail(PP_EINVAL, "h, w must be >= 1");
  const long hn = h + 2L * v.pad - 2L * v.dil - 1, wn = w + 2L * v.pad - 2L * v.dil - 1;
  if (hn < 0 || wn < 0) return fail(PP_EINVAL, "input smaller than the dilated kernel");
  if (h_out) *h_out = static_cast<int32_t>(hn / v.stride + 1);
  if (w_out) *w_out = static_cast<int32_t>(wn / v.stride + 1);
  return PP_OK;
}

extern "C" pp_status pp_conv2d_recipe(const void* h_blob, size_t blob_bytes, int32_t n, int32_t h, int32_t w,
                                      int32_t act_dtype, int32_t with_workspace, int32_t* recipe, int32_t* ksplit) {
  clear_error();
  BlobView v;
  pp_status s = parse_blob(h_blob, blob_bytes, &v, /*full=*/false);
  if (s != PP_OK) return s;
  if (!recipe) return fail(PP_EINVAL, "recipe is NULL");
  int ho = 0, wo = 0;
  s = conv_check(v, n, h, w, act_dtype, &ho, &wo);
  if (s != PP_OK) return s;
  const ConvParams p = layer_params(v, n, h, w, ho, wo);
  ConvPlan plan = plan_conv(p, library_kind(v), act_dtype == PP_BF16, with_workspace != 0);
  if (library_kind(v) == kLibGeneric && jit_library4(v)) {
    // with run-time compiled kernels the call runs the canonical library's plan
    const ConvPlan cp = plan_conv(p, kLibCanon8, act_dtype == PP_BF16, with_workspace != 0, true);
    if (cp.recipe >= 0 && jit_ready(v, cp, act_dtype == PP_BF16)) plan = cp;
  }
  *recipe = plan.recipe;
  if (ksplit) *ksplit = plan.ksplit;
  return PP_OK;
}

extern "C" pp_status pp_jit_library(const void* h_blob, size_t blob_bytes, int32_t n, int32_t h, int32_t w,
                                    int32_t act_dtype, int32_t with_workspace) {
  clear_error();
  BlobView v;
  pp_status s = parse_blob(h_blob, blob_bytes, &v, /*full=*/false);
  if (s != PP_OK) return s;
  int ho = 0, wo = 0;
  s = conv_check(v, n, h, w, act_dtype, &ho, &wo);
  if (s != PP_OK) return s;
  if (!jit_library4(v))
    return fail(PP_EUNSUPPORTED, "run-time kernels are for libraries of up to 8 four-tap patterns other than the "
                                 "canonical one");
  if (v.pad != v.dil) return fail(PP_EUNSUPPORTED, "run-time kernels need pad = dilation");
  const ConvParams p = layer_params(v, n, h, w, ho, wo);
  const bool bf = act_dtype == PP_BF16;
  // the plans pp_conv2d_fwd can make: with the workspace's split, and without
  for (bool split : {with_workspace != 0, false}) {
    const ConvPlan plan = plan_conv(p, kLibCanon8, bf, split, true);
    if (plan.recipe < 0) return fail(PP_EUNSUPPORTED, "no tiling runs this layer");
    if (plan.recipe == kRecipeMfma) continue;   // the matrix-core form reads any library from the blob
    s = jit_prepare(v, plan, bf);
    if (s != PP_OK) return s;
  }
  return PP_OK;
}

extern "C" pp_status pp_conv2d_workspace(const void* h_blob, size_t blob_bytes, int32_t n, int32_t h, int32_t w,
                                         int32_t act_dtype, size_t* bytes) {
  clear_error();
  BlobView v;
  pp_status s = parse_blob(h_blob, blob_bytes, &v, /*full=*/false);
  if (s != PP_OK) return s;
  if (!bytes) return fail(PP_EINVAL, "bytes is NULL");
  int ho = 0, wo = 0;
  s = conv_check(v, n, h, w, act_dtype, &ho, &wo);
  if (s != PP_OK) return s;
  *bytes = conv_scratch_bytes(v, n, h, w, act_dtype);
  if (library_kind(v) == kLibGeneric && jit_library4(v)) {
    // enough for the canonical plan that run-time compiled kernels run
    const ConvParams p = layer_params(v, n, h, w, ho, wo);
    const size_t b = split_bytes(plan_conv(p, kLibCanon8, act_dtype == PP_BF16, true, true), p);
    if (b > *bytes) *bytes = b;
  }
  return PP_OK;
}

namespace pp {
// a layer's prepared weights: the bf16 matrix-core form's (bf16 layers it
// serves: c_in a multiple of 32), then, from the next 256-byte boundary, the
// lean kernel's fp32 expansion (canonical library, pad = dilation, stride
// and dilation 1; fp32 also stride 1 with dilation 2 and stride 2 with
// dilation 1; fp32 or bf16 weights); either part may be absent
static bool mfma_part(const BlobView& v, const ConvParams& p) { return v.wdtype == PP_BF16 && mfma_eligible(p); }
static bool lean_part(const BlobView& v) {
  const bool f32 = v.wdtype == PP_F32;
  return library_kind(v) == kLibCanon8 && v.pad == v.dil &&
         ((v.stride == 1 && v.dil == 1) || (f32 && ((v.stride == 1 && v.dil == 2) || (v.stride == 2 && v.dil == 1))));
}
static size_t lean_part_offset(const BlobView& v, const ConvParams& p) {
  return mfma_part(v, p) ? align256(mfma_bytes(p)) : 0;
}

size_t prepared_bytes(const BlobView& v) {
  const ConvParams p = layer_params(v, 1, 3 * v.dil, 3 * v.dil, 1, 1);
  if (!lean_part(v)) return mfma_part(v, p) ? mfma_bytes(p) : 0;
  return lean_part_offset(v, p) + lean_prepared_bytes(p);
}

const void* lean_prepared(const BlobView& v, const void* prepared) {
  if (!prepared || !lean_part(v)) return nullptr;
  const ConvParams p = layer_params(v, 1, 3 * v.dil, 3 * v.dil, 1, 1);
  return static_cast<const uint8_t*>(prepared) + lean_part_offset(v, p);
}

static bool preparable(const BlobView& v, const ConvParams& p) { return mfma_part(v, p) || lean_part(v); }
}  // namespace pp

extern "C" pp_status pp_conv2d_prepare(const void* h_blob, size_t blob_bytes, const void* d_blob, void* prepared,
                                       size_t* inout_bytes, void* hip_stream) {
  clear_error();
  BlobView v;
  pp_status s = parse_blob(h_blob, blob_bytes, &v, /*full=*/false);
  if (s != PP_OK) return s;
  if (!inout_bytes) return fail(PP_EINVAL, "inout_bytes is NULL");
  // the expansion does not depend on the input size: one pixel stands in
  ConvParams p = layer_params(v, 1, 3 * v.dil, 3 * v.dil, 1, 1);
  if (!preparable(v, p))
    return fail(PP_EUNSUPPORTED, v.wdtype == PP_BF16 ? "bf16 prepared weights need c_in a multiple of 32 (the "
                                                       "matrix-core form) or the canonical library with stride 1, "
                                                       "dilation 1 and pad 1 (the lean kernel)"
                                                     : "fp32 prepared weights need the canonical library, pad = "
                                                       "dilation, and stride and dilation 1, or one of them 2");
  const size_t need = prepared_bytes(v);
  if (!prepared) {
    *inout_bytes = need;
    return PP_OK;
  }
  if (*inout_bytes < need) {
    *inout_bytes = need;
    return fail(PP_ESIZE, "prepared buffer too small");
  }
  if (!d_blob || reinterpret_cast<uintptr_t>(d_blob) % 256 || reinterpret_cast<uintptr_t>(prepared) % 256)
    return fail(PP_EINVAL, "d_blob and prepared must be 256-byte aligned device pointers");
  p.blob = static_cast<const uint8_t*>(d_blob);
  const hipStream_t st = static_cast<hipStream_t>(hip_stream);
  hipError_t e = hipSuccess;
  if (mfma_part(v, p)) e = launch_mfma_expand(p, prepared, st);
  if (e == hipSuccess && lean_part(v))
    e = launch_lean_expand(p, v.wdtype == PP_BF16, static_cast<uint8_t*>(prepared) + lean_part_offset(v, p), st);
  if (e != hipSuccess) return fail(PP_EHIP, std::string("expansion launch: ") + hipGetErrorString(e));
  return PP_OK;
}

extern "C" pp_status pp_conv2d_fwd(const void* h_blob, size_t blob_bytes, const void* d_blob, const void* x,
                                   void* y, int32_t n, int32_t h, int32_t w, int32_t act_dtype, uint32_t flags,
                                   void* workspace, size_t ws_bytes, void* hip_stream) {
  clear_error();
  BlobView v;
  pp_status s = parse_blob(h_blob, blob_bytes, &v, /*full=*/false);
  if (s != PP_OK) return s;
  if (ws_bytes && !workspace) return fail(PP_EINVAL, "NULL workspace with nonzero size");
  return conv_enqueue(v, d_blob, x, y, n, h, w, act_dtype, flags, workspace, workspace ? ws_bytes : 0,
                      static_cast<hipStream_t>(hip_stream));
}
