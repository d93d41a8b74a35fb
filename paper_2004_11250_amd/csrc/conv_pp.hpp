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
  uint32_t blob_bytes = 0;  // total bytes of the blob (its buffer resource bound)
  uint32_t n_wt = 0;        // weight elements; every weight offset read from the device is clamped to it
  int n_patterns = 0;
  uint32_t flags = 0;
  int tiles_x = 0, tiles_y = 0, n_ftiles = 0;   // filled by the launcher
};

// The compiled tilings ("recipes"):
//   id, R x CC outputs per lane, LW lanes across (64/LW down), WF filter waves
//   (8 filters each), WS channel-split waves, CPW channels per wave per chunk.
#define PP_RECIPES(X)       \
  X(0, 4, 4, 8, 1, 4, 1)    \
  X(1, 4, 4, 8, 2, 2, 2)    \
  X(2, 4, 4, 8, 4, 1, 4)    \
  X(3, 2, 4, 8, 1, 4, 2)    \
  X(4, 2, 4, 8, 2, 2, 4)    \
  X(5, 2, 4, 8, 4, 1, 8)    \
  X(6, 2, 2, 8, 1, 4, 4)    \
  X(7, 2, 2, 8, 2, 2, 8)    \
  X(8, 2, 2, 8, 1, 8, 2)    \
  X(9, 1, 2, 8, 1, 8, 2)    \
  X(10, 1, 1, 8, 1, 8, 2)   \
  X(11, 4, 2, 8, 1, 4, 2)   \
  X(12, 2, 4, 8, 1, 4, 1)   \
  X(13, 2, 2, 8, 1, 4, 1)   \
  X(14, 2, 4, 8, 8, 1, 8)   \
  X(15, 2, 2, 8, 4, 1, 8)   \
  X(16, 2, 2, 8, 4, 2, 4)   \
  X(17, 2, 4, 8, 4, 2, 4)   \
  X(18, 4, 4, 8, 2, 1, 4)   \
  X(19, 2, 2, 8, 2, 4, 4)

constexpr int kNumRecipes = 20;

struct RecipeInfo {
  int r, cc, lw, wf, ws, cpw;
};

// geometry of a recipe, and whether its LDS footprint fits for (stride, dilation)
RecipeInfo recipe_info(int id);
bool recipe_fits(int id, int stride, int dil, bool bf16, int lib);
// recipes compiled for a pattern library (the canonical library gets all)
bool recipe_compiled(int lib, int id);

struct ConvPlan {
  int recipe = 0;
};

ConvPlan plan_conv(const ConvParams& p, int lib, bool bf16);
hipError_t launch_conv(int lib, const ConvPlan& plan, const ConvParams& p, bool bf16_act, hipStream_t st);

template <int LIB, int S, int D, class TA>
hipError_t launch_recipe(int id, const ConvParams& p, hipStream_t st);

}  // namespace pp
