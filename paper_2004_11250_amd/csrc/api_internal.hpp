// api_internal.hpp -- helpers shared by the C-ABI entry points.
#pragma once

#include <hip/hip_runtime.h>

#include "ppk1.hpp"

namespace pp {

// kLibCanon8 / kLibDense9 / kLibGeneric for a parsed blob's pattern library
int library_kind(const BlobView& v);

// validate shapes of a pruned conv; returns the output size
pp_status conv_check(const BlobView& v, int32_t n, int32_t h, int32_t w, int32_t act_dtype, int* ho, int* wo);

// validate pointers and enqueue one pruned conv on `st`
pp_status conv_enqueue(const BlobView& v, const void* d_blob, const void* x, void* y, int32_t n, int32_t h,
                       int32_t w, int32_t act_dtype, uint32_t flags, hipStream_t st);

}  // namespace pp
