// conv_pp.hpp -- launch interface of the pruned 3x3 convolution kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "pp.h"

namespace pp {

enum { kLibGeneric = 0, kLibCanon8 = 1, kLibDense9 = 2 };

// Everything a launch needs; offsets are byte offsets into the device blob.
struct ConvParams {
  const uint8_t* blob = nullptr;
  const void* x = nullptr;
  void* y = nullptr;
  int n = 0, h = 0, w = 0, ho = 0, wo = 0;
  int c_in = 0, c_out = 0, pad = 0, stride = 1, dil = 1, n_groups = 0;
  uint32_t off_codes = 0, off_woff = 0, off_w = 0, off_bias = 0, off_perm = 0, off_masks = 0;
  uint32_t n_wt = 0;        // weight elements; every weight offset read from the device is clamped to it
  int n_patterns = 0;
  uint32_t flags = 0;
  int tiles_x = 0, tiles_y = 0, n_ftiles = 0;   // filled by the launcher
};

// Which compiled tiling to use for a layer shape.
struct ConvPlan {
  int recipe = 0;
};

ConvPlan plan_conv(const ConvParams& p, int lib);
hipError_t launch_conv(int lib, const ConvPlan& plan, const ConvParams& p, bool bf16_act, hipStream_t st);

}  // namespace pp
