// api_internal.hpp -- helpers shared by the C-ABI entry points.
#pragma once

#include <hip/hip_runtime.h>

#include "conv_pp.hpp"
#include "ppk1.hpp"

namespace pp {

// kLibCanon8 / kLibDense9 / kLibGeneric for a parsed blob's pattern library
int library_kind(const BlobView& v);

// validate shapes of a pruned conv; returns the output size
pp_status conv_check(const BlobView& v, int32_t n, int32_t h, int32_t w, int32_t act_dtype, int* ho, int* wo);

// validate pointers and enqueue one pruned conv on `st`.  scratch (may be
// NULL) of scratch_bytes lets the planner split the input channels over
// workgroups (partial sums there, added by a second kernel)
// wprep: an fp32 layer's prepared lean weights (or null), read when the plan
// is a lean tiling built for them; the scratch then still serves a split
pp_status conv_enqueue(const BlobView& v, const void* d_blob, const void* x, void* y, int32_t n, int32_t h,
                       int32_t w, int32_t act_dtype, uint32_t flags, void* scratch, size_t scratch_bytes,
                       hipStream_t st, const void* wprep = nullptr);

// whether pp_conv2d_fwd can fuse the ops before / after the conv (flags:
// PP_UPSAMPLE2 and one of PP_MAXPOOL2, PP_ACCUMULATE, PP_PIXSHUF2) for this
// layer, with or without split scratch; h, w: the conv's input size (with
// PP_UPSAMPLE2 the upsampled size)
bool conv_fusable(const BlobView& v, int32_t n, int32_t h, int32_t w, int32_t act_dtype, uint32_t flags,
                  bool with_scratch);

// run-time specialised kernels (jit.cpp): whether the layer's library is
// one of up to 8 four-tap patterns other than the canonical one; compile the
// kernel(s) of a plan (made as for the canonical library) for the current
// device; launch them if compiled (false: not compiled, nothing launched)
bool jit_library4(const BlobView& v);
pp_status jit_prepare(const BlobView& v, const ConvPlan& plan, bool bf16);
bool jit_ready(const BlobView& v, const ConvPlan& plan, bool bf16);
bool jit_launch(const BlobView& v, const ConvPlan& plan, ConvParams p, bool bf16, hipStream_t st, hipError_t* err);

// the plan of a layer whose channel split may use scratch_bytes of scratch
// (a plan whose split needs more runs unsplit)
ConvPlan plan_with_scratch(const ConvParams& p, int kind, bool bf16, size_t scratch_bytes, bool no_lean);

// the tiling pp_conv2d_fwd runs for this layer (flags as there; h, w: the
// stored input size) with scratch_bytes of split scratch; -1 if none
int conv_recipe(const BlobView& v, int32_t n, int32_t h, int32_t w, int32_t act_dtype, uint32_t flags,
                size_t scratch_bytes);

// bytes of a layer's prepared weights (pp_conv2d_prepare), and where in them
// the lean kernel's part starts (NULL: the layer has none)
size_t prepared_bytes(const BlobView& v);
const void* lean_prepared(const BlobView& v, const void* prepared);

// scratch bytes pp_conv2d_fwd can use for this layer and input (0: none)
size_t conv_scratch_bytes(const BlobView& v, int32_t n, int32_t h, int32_t w, int32_t act_dtype);

}  // namespace pp
