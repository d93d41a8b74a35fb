// dense.hpp -- launch interface of the dense and glue kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace pp {

struct DenseParams {
  const void* x = nullptr;
  void* y = nullptr;
  const void* wt = nullptr;     // weights in the activation dtype
  const float* bias = nullptr;  // fp32 or NULL
  int n = 0, c_in = 0, h = 0, w = 0, c_out = 0, ho = 0, wo = 0;
  int k = 0, stride = 1, pad = 0;
  int relu = 0;
  // transposed conv: device scratch of deconv_scratch_bytes() for the
  // weights laid out per parity class (or NULL: read them as given)
  void* scratch = nullptr;
};

enum { kGlueMaxPool2 = 0, kGlueUp2 = 1, kGluePixShuf2 = 2, kGlueAdd = 3 };

struct GlueParams {
  int op = 0;
  const void* x = nullptr;
  const void* x2 = nullptr;
  void* y = nullptr;
  int n = 0, c_in = 0, h = 0, w = 0, c_out = 0, ho = 0, wo = 0;
};

hipError_t launch_dense_conv(const DenseParams& p, bool bf16, hipStream_t st);
hipError_t launch_deconv(const DenseParams& p, bool bf16, hipStream_t st);
size_t deconv_scratch_bytes(int c_in, int c_out, bool bf16);
hipError_t launch_glue(const GlueParams& p, bool bf16, hipStream_t st);

}  // namespace pp
