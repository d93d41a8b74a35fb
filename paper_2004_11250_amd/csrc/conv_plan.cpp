// conv_plan.cpp -- choice of tiling ("recipe") for a pruned 3x3 layer and
// dispatch to the compiled kernels.
#include <cstdlib>

#include "conv_pp.hpp"

namespace pp {

RecipeInfo recipe_info(int id) {
  switch (id) {
#define PP_X(ID, R, CC, LW, WF, WS, CPW) \
  case ID:                               \
    return RecipeInfo{R, CC, LW, WF, WS, CPW};
    PP_RECIPES(PP_X)
#undef PP_X
  }
  return RecipeInfo{0, 0, 0, 0, 0, 0};
}

// same LDS accounting as the kernel (Geo in conv_pp_kernel.hpp): fp32 uses
// double-buffered DMA staging with 64*NW-float channel regions, and the
// canonical library also stages its group data (metadata + weights)
bool recipe_fits(int id, int s, int d, bool bf16, int lib) {
  const RecipeInfo r = recipe_info(id);
  if (r.r == 0) return false;
  const int lh = 64 / r.lw;
  const int th = lh * r.r, tw = r.lw * r.cc;
  const int tih = (th - 1) * s + 2 * d + 1, tiw = (tw - 1) * s + 2 * d + 1;
  const int lstr = (tiw + 3) / 4 * 4;
  const int nw = r.wf * r.ws, cch = r.ws * r.cpw;
  const bool dma = !bf16;
  const bool ldsw = dma && lib == kLibCanon8;
  const int seg = 64 * nw;
  const int chstr = dma ? (tih * lstr + seg - 1) / seg * seg : tih * lstr;
  const long gdata = ldsw ? static_cast<long>(r.wf) * cch * 32 : 0;
  const long meta = ldsw ? 4L * r.wf * 64 : 0;
  const long buf = static_cast<long>(cch) * chstr + gdata;
  const long red = r.ws > 1 ? static_cast<long>(r.ws / 2) * r.wf * 8 * r.r * r.cc * 64 : 0;
  const long total = (buf > red ? buf : red) + (dma ? buf : 0) + meta;
  return total * 4 <= 160 * 1024 && cch <= 16 && cch % 2 == 0;
}

bool recipe_compiled(int lib, int id) {
  return lib == kLibCanon8 || id == 0 || id == 3 || id == 6 || id == 8 || id == 12 || id == 13;
}

static int env_recipe() {
  const char* e = std::getenv("PP_RECIPE");
  if (!e || !*e) return -1;
  return std::atoi(e);
}

ConvPlan plan_conv(const ConvParams& p, int lib, bool bf16) {
  ConvPlan plan;
  const int forced = env_recipe();
  if (forced >= 0 && forced < kNumRecipes && recipe_compiled(lib, forced) && recipe_fits(forced, p.stride, p.dil, bf16, lib)) {
    plan.recipe = forced;
    return plan;
  }
  const long pix = static_cast<long>(p.ho) * p.wo;
  int pref[4];
  if (lib == kLibCanon8 && !bf16 && p.stride == 1) {
    // fp32 canonical library, from timings of every tiling on the VGG-16
    // layer shapes (MI355X)
    if (pix >= 160L * 160L) {
      pref[0] = 17; pref[1] = 16; pref[2] = 4; pref[3] = 13;
    } else if (pix >= 80L * 80L) {
      pref[0] = 19; pref[1] = 3; pref[2] = 13; pref[3] = 13;
    } else if (pix >= 20L * 20L) {
      pref[0] = 8; pref[1] = 19; pref[2] = 6; pref[3] = 13;
    } else {
      pref[0] = 10; pref[1] = 9; pref[2] = 8; pref[3] = 13;
    }
  } else if (pix >= 100L * 100L) {
    pref[0] = 0; pref[1] = 3; pref[2] = 12; pref[3] = 13;
  } else if (pix >= 40L * 40L) {
    pref[0] = 3; pref[1] = 12; pref[2] = 13; pref[3] = 13;
  } else if (pix >= 20L * 20L) {
    pref[0] = 6; pref[1] = 13; pref[2] = 13; pref[3] = 13;
  } else {
    pref[0] = 8; pref[1] = 13; pref[2] = 13; pref[3] = 13;
  }
  for (int id : pref)
    if (recipe_compiled(lib, id) && recipe_fits(id, p.stride, p.dil, bf16, lib)) {
      plan.recipe = id;
      return plan;
    }
  plan.recipe = 13;
  return plan;
}

template <int LIB, class TA>
static hipError_t launch_lib(int id, const ConvParams& p, hipStream_t st) {
  if (p.stride == 1 && p.dil == 1) return launch_recipe<LIB, 1, 1, TA>(id, p, st);
  if (p.stride == 2 && p.dil == 1) return launch_recipe<LIB, 2, 1, TA>(id, p, st);
  if (p.stride == 1 && p.dil == 2) return launch_recipe<LIB, 1, 2, TA>(id, p, st);
  if (p.stride == 2 && p.dil == 2) return launch_recipe<LIB, 2, 2, TA>(id, p, st);
  return hipErrorInvalidValue;
}

hipError_t launch_conv(int lib, const ConvPlan& plan, const ConvParams& p, bool bf16_act, hipStream_t st) {
  if (!recipe_compiled(lib, plan.recipe) || !recipe_fits(plan.recipe, p.stride, p.dil, bf16_act, lib))
    return hipErrorInvalidConfiguration;
  if (bf16_act) {
    if (lib == kLibCanon8) return launch_lib<kLibCanon8, uint16_t>(plan.recipe, p, st);
    if (lib == kLibDense9) return launch_lib<kLibDense9, uint16_t>(plan.recipe, p, st);
    return launch_lib<kLibGeneric, uint16_t>(plan.recipe, p, st);
  }
  if (lib == kLibCanon8) return launch_lib<kLibCanon8, float>(plan.recipe, p, st);
  if (lib == kLibDense9) return launch_lib<kLibDense9, float>(plan.recipe, p, st);
  return launch_lib<kLibGeneric, float>(plan.recipe, p, st);
}

}  // namespace pp
