// conv_plan.cpp -- choice of tiling ("recipe") for a pruned 3x3 layer and
// dispatch to the compiled kernels.
#include <algorithm>
#include <cmath>
#include <cstdlib>

#include "conv_pp.hpp"

namespace pp {

RecipeInfo recipe_info(int id) {
  switch (id) {
#define PP_X(ID, R, CC, LW, WF, WS, CPW) \
  case ID:                               \
    return RecipeInfo{R, CC, LW, WF, WS, CPW, 0};
    PP_RECIPES(PP_X)
#undef PP_X
#define PP_W(ID, R, CC, LW, WS, P) \
  case ID:                         \
    return RecipeInfo{R, CC, LW, 1, WS, 0, P};
    PP_WRECIPES(PP_W)
#undef PP_W
#define PP_L(ID, R, CC, LW, WS, V4) \
  case ID:                          \
    return RecipeInfo{R, CC, LW, 1, WS, 0, 0};
    PP_LRECIPES(PP_L)
#undef PP_L
  }
  return RecipeInfo{0, 0, 0, 0, 0, 0, 0};
}

static bool is_wave_recipe(int id) { return id >= kFirstWaveRecipe && id < kNumRecipes; }

// LDS accounting of the wave-pipeline kernel (shared with WGeo in conv_pp_wave.hpp)
static bool wave_recipe_fits(const RecipeInfo& r, int s, int d, int lib, bool bf16) {
  const int warea = lib == kLibDense9 ? 128 : 64;
  return wave_lds_floats(r.r, r.cc, r.lw, r.ws, s, d, warea, bf16) * 4 <= 160 * 1024 && r.ws >= 1 && r.ws <= 16;
}

bool recipe_fits(int id, int s, int d, bool bf16, int lib) {
  const RecipeInfo r = recipe_info(id);
  if (r.r == 0) return false;
  if (is_lean_recipe(id)) return lib == kLibCanon8 && lean_lds_bytes(id, bf16, d, s) > 0;
  if (is_wave_recipe(id)) return (lib == kLibCanon8 || lib == kLibDense9) && wave_recipe_fits(r, s, d, lib, bf16);
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
  if (is_lean_recipe(id)) return lib == kLibCanon8;
  if (id < 0 || id >= kNumRecipes) return false;
  if (is_wave_recipe(id)) return lib == kLibCanon8 || lib == kLibDense9;
  return lib == kLibCanon8 || id == 0 || id == 3 || id == 6 || id == 8 || id == 12 || id == 13;
}

// a recipe that can run this layer: compiled for the library, fits in LDS,
// (wave-pipeline kernel) compiled for the layer's padding (pad = dilation),
// and (register-pipelined tilings) fp32 with the canonical library
static bool recipe_usable(int id, const ConvParams& p, int lib, bool bf16) {
  if (!recipe_compiled(lib, id) || !recipe_fits(id, p.stride, p.dil, bf16, lib)) return false;
  if (is_lean_recipe(id)) {
    if (bf16 && (p.w % 2 != 0 || (p.flags & (PP_UPSAMPLE2 | PP_PIXSHUF2)))) return false;
    if ((p.dil != 1 || p.stride != 1) && (p.flags & PP_UPSAMPLE2)) return false;
    return p.pad == p.dil && (!lean_v4(id) || (p.w % (bf16 ? 8 : 4) == 0 && !(p.flags & PP_UPSAMPLE2)));
  }
  if (recipe_info(id).pipe && (bf16 || lib != kLibCanon8)) return false;
  return !is_wave_recipe(id) || p.pad == p.dil;
}

static int env_recipe() {
  const char* e = std::getenv("PP_RECIPE");
  if (!e || !*e) return -1;
  return std::atoi(e);
}

static int env_int(const char* name) {
  const char* e = std::getenv(name);
  if (!e || !*e) return -1;
  return std::atoi(e);
}

// output tiles of a recipe for this layer
static long tiles_of(int id, const ConvParams& p) {
  const RecipeInfo r = recipe_info(id);
  const long th = (64 / r.lw) * r.r, tw = static_cast<long>(r.lw) * r.cc;
  return ((p.ho + th - 1) / th) * ((p.wo + tw - 1) / tw);
}

// waves of a wave-pipeline recipe's grid (no split)
static long waves_of(int id, const ConvParams& p) {
  return static_cast<long>(p.n) * tiles_of(id, p) * p.n_groups * recipe_info(id).ws;
}

// channel split of a wave-pipeline recipe: only for grids of at most one
// wave per SIMD (1024 waves), up to about 4 waves per SIMD, keeping at least
// 8 channels per wave (measured on MI355X: splitting grids that already hold
// 1.5-2 waves per SIMD costs more in partial sums than it gains, except for
// the 16-wave 1 x 2 tilings on the 14 x 14 layers, where 2 splits of 2048
// waves beat both no split and the 8-wave tilings split 4 ways)
static int choose_split(int id, const ConvParams& p) {
  const RecipeInfo r = recipe_info(id);
  const long items = static_cast<long>(p.n) * tiles_of(id, p) * p.n_groups;
  const long waves = items * r.ws;
  int ks = 1;
  if (waves <= (r.ws == 16 && r.r == 1 ? 2048 : 1024))
    while (waves * ks * 2 <= 4096 && static_cast<long>(p.c_in) / (ks * 2) >= 8L * r.ws) ks *= 2;
  const int forced = env_int("PP_KSPLIT");
  if (forced >= 1) ks = forced < p.c_in ? forced : p.c_in;
  return ks;
}

// channel split of a lean tiling: the 16-wave tilings on maps of at most
// 16 x 16 outputs run split, the one-row-per-lane ones two ways and the 2 x 2
// ones four ways, keeping at least 8 channels per wave (measured on MI355X
// at 14 x 14, 512 -> 512: 2 x 2 split four ways 18 us, one row split two
// ways 19 us, unsplit 26-28 us); none on larger maps, where the grid already
// holds four waves per SIMD and a split only adds partial sums
static int choose_split_lean(int id, const ConvParams& p) {
  const int forced = env_int("PP_KSPLIT");
  if (forced >= 1) return forced < p.c_in ? forced : p.c_in;
  const RecipeInfo r = recipe_info(id);
  if (r.ws != 16 || static_cast<long>(p.ho) * p.wo > 16L * 16) return 1;
  int ks = r.r == 1 ? 2 : 4;
  while (ks > 1 && p.c_in / (ks * r.ws) < 8) ks /= 2;
  return ks;
}

static ConvPlan finish_plan(int id, const ConvParams& p, bool allow_split) {
  ConvPlan plan;
  plan.recipe = id;
  plan.ksplit = allow_split ? (is_wave_recipe(id) ? choose_split(id, p) : is_lean_recipe(id) ? choose_split_lean(id, p) : 1)
                            : 1;
  return plan;
}

size_t split_bytes(const ConvPlan& plan, const ConvParams& p) {
  if (plan.recipe == kRecipeMfma) return mfma_bytes(p);
  if (plan.ksplit <= 1) return 0;
  const RecipeInfo r = recipe_info(plan.recipe);
  const size_t items = static_cast<size_t>(p.n) * tiles_of(plan.recipe, p) * p.n_groups;
  return items * plan.ksplit * 8 * r.r * r.cc * 64 * sizeof(float);
}

// a fused 2 x 2 max pool is taken by the conv kernel when each lane holds
// whole windows (wave-pipeline tilings with even R and CC; tile origins are
// then even too), or by the second pass of a channel split, which sees whole
// tiles (every wave-pipeline tile is 8 R x 8 CC outputs: even)
static bool pool_fits(int id) {
  const RecipeInfo r = recipe_info(id);
  return (is_wave_recipe(id) || is_lean_recipe(id)) && r.r % 2 == 0 && r.cc % 2 == 0;
}

// whether the matrix-core form of a bf16 layer beats the vector kernels: a
// time model of each, its constants fitted to the bf16 layers of the five
// workloads on MI355X.  The wave-pipeline kernel does n_wt MACs per output
// pixel (n_wt: stored weights, about the surviving taps) at about 12 T MAC/s
// (half that at stride 2); the lean kernel (lean: it can run the layer) costs
// about one step per (output pixel, input channel, slot group), pruned slots
// all but free, plus 5 us, at a rate set by the tiling the lean table picks:
// about 1.0 T steps/s for the 4 x 4 tilings (maps from 160 x 160 up to
// 256 x 256 and from 512 x 512, or batches of 64 K outputs and more), 1.25 T
// for 2 x 4 on maps in between, 1.5 T on maps from 80 x 80, 1.1 T below (with prepared weights: VGG-16's layers 14-28 us, the style
// network's 128 -> 128 at 128 x 128 25.6 us).  The matrix-core form is
// latency-bound while the chip
// holds all its workgroups (about 1.4-1.5 us per k step, each waiting for
// its own loads), else bound by workgroup steps (about 880 / 390 per us for
// 64 / 128-filter tiles); plus about 8 us for the weight expansion and its
// launch.
static bool mfma_pays(const ConvParams& p, bool lean) {
  const double pix = static_cast<double>(p.n) * p.ho * p.wo;
  const double map = static_cast<double>(p.ho) * p.wo;
  const double lean_rate = p.n == 1 && map >= 256.0 * 256.0 && map < 512.0 * 512.0 ? 1.25e12
                           : (p.n > 1 ? pix >= 65536.0 : map >= 160.0 * 160.0) ? 1.0e12
                           : (p.n > 1 || map >= 80.0 * 80.0)                 ? 1.5e12
                                                                              : 1.1e12;
  const double t_vec = lean ? pix * p.c_in * p.n_groups / lean_rate + 5e-6
                            : pix * p.n_wt * (p.stride == 2 ? 2.2 : 1.0) / 12e12 + 8e-6;
  const bool long_k = mfma_long_k(p);
  const int km = long_k ? 64 : 32;
  const double steps = (9.0 * p.c_in + km - 1) / km;
  const long bm = p.c_out > 64 ? 128 : 64;
  const double wgs = std::ceil(pix / 128) * ((p.c_out + bm - 1) / bm);
  // (two wave groups per tile when the grid is at most one tile per compute
  // unit: about 0.8 of the latency-bound time)
  const double lat = steps * (long_k ? 1.5e-6 : 1.4e-6) * (wgs <= 256 ? 0.8 : 1.0);
  const double t_mfma = std::max(lat, wgs * steps / (bm == 128 ? 390e6 : 880e6)) + 8e-6;
  return t_mfma < t_vec;
}

ConvPlan plan_conv(const ConvParams& p, int lib, bool bf16, bool allow_split, bool no_lean) {
  const bool pool = (p.flags & PP_MAXPOOL2) != 0;
  // epilogues of the wave-pipeline kernel only
  const bool fused = (p.flags & (PP_MAXPOOL2 | PP_ACCUMULATE | PP_PIXSHUF2 | PP_UPSAMPLE2)) != 0;
  // a plan for recipe id, or recipe -1 when it cannot take the fused epilogue
  auto try_plan = [&](int id) {
    ConvPlan pl;
    pl.recipe = -1;
    if (no_lean && is_lean_recipe(id)) return pl;
    if (!recipe_usable(id, p, lib, bf16)) return pl;
    if (fused && !is_wave_recipe(id) && !is_lean_recipe(id)) return pl;
    pl = finish_plan(id, p, allow_split);
    if (pool && pl.ksplit == 1 && !pool_fits(id)) pl.recipe = -1;
    return pl;
  };
  const int forced = env_recipe();
  ConvPlan mfma;
  mfma.recipe = kRecipeMfma;
  const bool mfma_ok = bf16 && allow_split && mfma_eligible(p);
  if (forced == kRecipeMfma && mfma_ok) return mfma;
  ConvPlan cin;
  cin.recipe = kRecipeCin;
  const bool cin_ok = !no_lean && cin_eligible(p, bf16);
  if (forced == kRecipeCin && cin_ok) return cin;
  ConvPlan few;
  few.recipe = kRecipeFewOut;
  const bool few_any = !no_lean && fewout_eligible(p);
  if (forced == kRecipeFewOut && few_any) return few;
  if (forced >= 0 && (forced < kNumRecipes || is_lean_recipe(forced))) {
    const ConvPlan pl = try_plan(forced);
    if (pl.recipe >= 0) return pl;
  }
  if (cin_ok && forced < 0) return cin;
  // (bf16: 64 -> 3 at 1080 x 1920 228 -> 135 us; fp32 stays on the wave kernel, 173 against 186 here)
  if (few_any && lib == kLibDense9 && bf16 && forced < 0) return few;
  // (dilation 2 = pad 2, or stride 2: fp32 only)
  const bool lean_layer = lib == kLibCanon8 && p.pad == p.dil &&
                          ((p.stride == 1 && p.dil == 1) ||
                           (!bf16 && ((p.stride == 1 && p.dil == 2) || (p.stride == 2 && p.dil == 1)))) &&
                          p.c_in > 8 && !no_lean;
  if (mfma_ok && forced < 0 &&
      mfma_pays(p, lean_layer && bf16 && p.w % 2 == 0 && !(p.flags & (PP_UPSAMPLE2 | PP_PIXSHUF2))))
    return mfma;
  const long pix = static_cast<long>(p.ho) * p.wo;
  if (lean_layer) {
    // fp32, stride 1: the lean tilings that timed fastest on the
    // VGG-16 layer shapes (MI355X), by output size: 4 x 4 outputs per lane on
    // the 224 x 224 maps (4 channel-split waves), 2 x 4 on 112 x 112 (8
    // waves) and 56 x 56 (16 waves, two-channel rings), 2 x 2 with 16 waves
    // on 28 x 28 and, with 4-byte staging and a channel split, on smaller
    // maps (else one row of 2 outputs per lane).  Each 16-byte staging tiling has a
    // 4-byte staging twin of the same tiling (widths not a multiple of 4, a
    // fused x2 upsample): same accumulation order, so a conv fused with the
    // upsample before it gives bitwise what the unfused conv gives.
    // Batches (timed on the colourization layer shapes, 8 images): 2 x 4
    // outputs per lane with 8 waves up to 8 x 64 x 64 outputs (512 -> 512 at
    // 32 x 32: 162 us against 220 on the wave kernel), 4 x 4 beyond.
    // Dilation 2 (fp32; the colourization network's 512 -> 512 at 32 x 32,
    // 8 images): 4 x 4 outputs per lane with 4-byte staging, whose smaller
    // LDS tile fits two workgroups per CU (130 us against 186 for 2 x 4 and
    // 192 on the wave kernel).
    int lp[4] = {-1, -1, -1, -1};
    if (p.stride == 2) {
      lp[0] = 49; lp[1] = 53;
    } else if (p.dil == 2) {
      lp[0] = 56; lp[1] = 55;
    } else if (p.n > 1) {
      if (static_cast<long>(p.n) * pix >= 65536L) {
        lp[0] = 40; lp[1] = 56;
      } else {
        lp[0] = 46; lp[1] = 55;
      }
    } else if (pix >= 256L * 256L && pix < 512L * 512L) {
      // (super-resolution 64 -> 64 at 270 x 480: 2 x 4 58.6 us against 74
      // for 4 x 4; its 64 -> 256 at 540 x 960: 4 x 4 874 us against 949)
      lp[0] = 46; lp[1] = 55;
    } else if (pix >= 160L * 160L) {
      lp[0] = 40; lp[1] = 56;
    } else if (pix >= 80L * 80L) {
      lp[0] = 46; lp[1] = 55;
    } else if (pix >= 40L * 40L) {
      lp[0] = 58; lp[1] = 59;
    } else if (pix >= 20L * 20L) {
      lp[0] = 48; lp[1] = 51;
    } else {
      lp[0] = 51; lp[1] = 54;
    }
    if (forced < 0)
      for (int id : lp)
        if (id >= 0) {
          const ConvPlan pl = try_plan(id);
          if (pl.recipe >= 0) return pl;
        }
  }
  int pref[4];
  const bool wave_ok = (lib == kLibCanon8 || lib == kLibDense9) && p.pad == p.dil;
  if (wave_ok && !bf16 && p.stride == 1 && p.n == 1) {
    // fp32, stride 1, one image: the wave-pipeline tilings that timed fastest
    // on the VGG-16 and super-resolution layer shapes (MI355X), by output
    // size; v4 tilings as fallback.  The register-pipelined tilings (32-34,
    // about 200 registers: two waves per SIMD) win while the whole grid is
    // resident at once (<= 2048 waves), and lose beyond that.
    if (lib == kLibDense9 || p.c_in <= 8) {
      pref[0] = 31; pref[1] = 20; pref[2] = 0; pref[3] = 13;
    } else if (pix >= 160L * 160L) {
      const long items31 = static_cast<long>(p.n) * tiles_of(31, p) * p.n_groups;
      if (static_cast<long>(p.n) * tiles_of(26, p) * p.n_groups <= 512) {
        // 4 x 4 outputs per lane: twice the FMAs per channel step for about
        // 1.3x its time, while its grid stays within two workgroups per CU
        pref[0] = 26; pref[1] = 32; pref[2] = 31; pref[3] = 30;
      } else if (waves_of(32, p) <= 2048) {
        pref[0] = 32; pref[1] = 31; pref[2] = 30; pref[3] = 17;
      } else if (items31 <= 4096) {
        pref[0] = 20; pref[1] = 31; pref[2] = 30; pref[3] = 17;
      } else {
        pref[0] = 31; pref[1] = 20; pref[2] = 30; pref[3] = 17;
      }
    } else if (pix >= 80L * 80L) {
      pref[0] = waves_of(33, p) <= 2048 ? 33 : 20; pref[1] = 20; pref[2] = 19; pref[3] = 3;
    } else if (pix >= 40L * 40L) {
      pref[0] = waves_of(34, p) <= 2048 ? 34 : 27; pref[1] = 27; pref[2] = 22; pref[3] = 8;
    } else if (pix >= 20L * 20L) {
      pref[0] = 23; pref[1] = 22; pref[2] = 8; pref[3] = 13;
    } else if (allow_split) {
      pref[0] = 38; pref[1] = 36; pref[2] = 24; pref[3] = 25;   // split 2 / 4 / 4 ways at 14 x 14
    } else {
      pref[0] = 25; pref[1] = 23; pref[2] = 10; pref[3] = 13;
    }
  } else if (wave_ok && !bf16 && lib == kLibCanon8 && p.c_in > 8) {
    // fp32 batches and strides 2 (timed on the style-transfer and
    // colourization layer shapes): 2 x 4 outputs per lane, two channel splits
    // per tile for very large grids, register-pipelined two- or four-way
    // splits for the smaller ones
    const long items = static_cast<long>(p.n) * tiles_of(31, p) * p.n_groups;
    if (items >= 4096) {
      pref[0] = 31; pref[1] = 20; pref[2] = 13; pref[3] = 13;
    } else if (items >= 2048) {
      pref[0] = p.stride == 2 ? 32 : 20; pref[1] = 31; pref[2] = 20; pref[3] = 13;
    } else if (items >= 1024) {
      pref[0] = p.stride == 2 ? 32 : 33; pref[1] = 31; pref[2] = 20; pref[3] = 13;
    } else {
      pref[0] = 33; pref[1] = 20; pref[2] = 31; pref[3] = 13;
    }
  } else if (wave_ok && bf16 && lib == kLibCanon8 && p.stride == 1 && p.n == 1 && pix < 80L * 80L) {
    // bf16, one image, small maps (timed on the VGG-16 layer shapes): the
    // stride-1 fp32 choices without register pipelining
    if (pix >= 40L * 40L) {
      pref[0] = 27; pref[1] = 22; pref[2] = 23; pref[3] = 13;
    } else if (pix >= 20L * 20L) {
      pref[0] = 23; pref[1] = 22; pref[2] = 21; pref[3] = 13;
    } else if (allow_split) {
      pref[0] = 39; pref[1] = 24; pref[2] = 23; pref[3] = 13;   // split 2 / 4 / 4 ways at 14 x 14
    } else {
      pref[0] = 25; pref[1] = 23; pref[2] = 22; pref[3] = 13;
    }
  } else if (wave_ok) {
    // bf16, and the all-ones library (timed on the super-resolution and
    // colourization layer shapes): 2 x 4 outputs per lane; two channel
    // splits per tile for very large grids, else four; few input channels
    // (first layers) with 1 x 4 outputs per lane
    const long items = static_cast<long>(p.n) * tiles_of(31, p) * p.n_groups;
    if (p.c_in <= 8) {
      pref[0] = 29; pref[1] = 31; pref[2] = 13; pref[3] = 13;
    } else if (items >= 4096) {
      pref[0] = 31; pref[1] = 20; pref[2] = 13; pref[3] = 13;
    } else {
      pref[0] = 20; pref[1] = 31; pref[2] = 13; pref[3] = 13;
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
  for (int id : pref) {
    const ConvPlan pl = try_plan(id);
    if (pl.recipe >= 0) return pl;
  }
  if (fused) {
    // the fused layer's fallbacks (2 x 4, then 2 x 2 outputs per lane)
    for (int id : {31, 20, 27, 23, 22, 21, 28}) {
      const ConvPlan pl = try_plan(id);
      if (pl.recipe >= 0) return pl;
    }
    ConvPlan none;
    none.recipe = -1;   // no tiling can fuse the epilogue
    return none;
  }
  return finish_plan(13, p, allow_split);
}

template <int LIB, class TA>
static hipError_t launch_lib(int id, const ConvParams& p, hipStream_t st) {
  if (p.stride == 1 && p.dil == 1) return launch_recipe<LIB, 1, 1, TA>(id, p, st);
  if (p.stride == 2 && p.dil == 1) return launch_recipe<LIB, 2, 1, TA>(id, p, st);
  if (p.stride == 1 && p.dil == 2) return launch_recipe<LIB, 1, 2, TA>(id, p, st);
  if (p.stride == 2 && p.dil == 2) return launch_recipe<LIB, 2, 2, TA>(id, p, st);
  return hipErrorInvalidValue;
}

template <int LIB, class TA>
static hipError_t launch_wave(int id, const ConvParams& p, hipStream_t st) {
  if (p.stride == 1 && p.dil == 1) return launch_wave_recipe<LIB, 1, 1, TA>(id, p, st);
  if (p.stride == 2 && p.dil == 1) return launch_wave_recipe<LIB, 2, 1, TA>(id, p, st);
  if (p.stride == 1 && p.dil == 2) return launch_wave_recipe<LIB, 1, 2, TA>(id, p, st);
  if (p.stride == 2 && p.dil == 2) return launch_wave_recipe<LIB, 2, 2, TA>(id, p, st);
  return hipErrorInvalidValue;
}

hipError_t launch_conv(int lib, const ConvPlan& plan, const ConvParams& p0, bool bf16_act, hipStream_t st) {
  ConvParams p = p0;
  if (plan.recipe == kRecipeMfma) return bf16_act ? launch_mfma_conv(p, st) : hipErrorInvalidConfiguration;
  if (plan.recipe == kRecipeCin) return cin_eligible(p, bf16_act) ? launch_cin_conv(p, bf16_act, st) : hipErrorInvalidConfiguration;
  if (plan.recipe == kRecipeFewOut)
    return fewout_eligible(p) ? launch_fewout_conv(p, bf16_act, st) : hipErrorInvalidConfiguration;
  p.ksplit = plan.ksplit;
  if (plan.ksplit > 1 && !is_wave_recipe(plan.recipe) && !is_lean_recipe(plan.recipe))
    return hipErrorInvalidConfiguration;
  if (!recipe_usable(plan.recipe, p, lib, bf16_act)) return hipErrorInvalidConfiguration;
  if (is_lean_recipe(plan.recipe)) return launch_lean_recipe(plan.recipe, p, bf16_act, st);
  if (is_wave_recipe(plan.recipe)) {
    if (lib == kLibDense9)
      return bf16_act ? launch_wave<kLibDense9, uint16_t>(plan.recipe, p, st) : launch_wave<kLibDense9, float>(plan.recipe, p, st);
    return bf16_act ? launch_wave<kLibCanon8, uint16_t>(plan.recipe, p, st) : launch_wave<kLibCanon8, float>(plan.recipe, p, st);
  }
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
