// conv_pp.hpp -- launch interface of the pruned 3x3 convolution kernels.
#pragma once

#ifndef __HIPCC_RTC__   // (the run-time compiler, which provides these itself)
#include <hip/hip_runtime.h>

#include <cstdint>
#endif

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
  // channel split over workgroups (wave-pipeline kernel): ksplit partial-sum
  // blocks per output tile in `part`, added by a second kernel
  int ksplit = 1;
  float* part = nullptr;
  // the lean kernel's prepared weights (fp32 canonical library): every
  // (slot group, channel)'s 8 slots x 4 taps expanded, zeros for pruned
  // slots, [n_groups][c_in][32] floats; null: the kernel stages them from
  // the blob itself
  const void* wprep = nullptr;
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

// Tilings of the wave-pipeline kernel (canonical library): id, R x CC
// outputs per lane, LW lanes across, WS channel-split waves of one slot group.
#define PP_WRECIPES(X)    \
  X(20, 2, 4, 8, 4, 0)    \
  X(21, 2, 2, 8, 4, 0)    \
  X(22, 2, 2, 8, 8, 0)    \
  X(23, 2, 2, 8, 16, 0)   \
  X(24, 1, 2, 8, 8, 0)    \
  X(25, 1, 1, 8, 16, 0)   \
  X(26, 4, 4, 8, 4, 0)    \
  X(27, 2, 4, 8, 8, 0)    \
  X(28, 2, 2, 8, 2, 0)    \
  X(29, 1, 4, 8, 2, 0)    \
  X(30, 1, 4, 8, 4, 0)    \
  X(31, 2, 4, 8, 2, 0)    \
  X(32, 2, 4, 8, 2, 1)    \
  X(33, 2, 4, 8, 4, 1)    \
  X(34, 2, 4, 8, 8, 1)    \
  X(35, 2, 2, 8, 8, 1)    \
  X(36, 1, 2, 8, 8, 1)    \
  X(37, 4, 4, 8, 2, 0)    \
  X(38, 1, 2, 8, 16, 1)   \
  X(39, 1, 2, 8, 16, 0)

constexpr int kFirstWaveRecipe = 20;

// Tilings of the lean kernel (fp32, canonical library, stride 1, pad 1): id,
// R x CC outputs per lane, LW lanes across, WS channel-split waves of one
// slot group, V4 16-byte staging (image width a multiple of 4; else 4-byte).
#define PP_LRECIPES(X)  \
  X(40, 4, 4, 8, 4, 1)  \
  X(41, 4, 4, 8, 2, 1)  \
  X(42, 4, 4, 8, 8, 1)  \
  X(43, 4, 4, 4, 4, 1)  \
  X(44, 4, 4, 4, 2, 1)  \
  X(45, 2, 4, 8, 4, 1)  \
  X(46, 2, 4, 8, 8, 1)  \
  X(47, 2, 2, 8, 8, 1)  \
  X(48, 2, 2, 8, 16, 1) \
  X(49, 2, 2, 8, 4, 1)  \
  X(50, 4, 4, 8, 1, 1)  \
  X(51, 2, 2, 8, 16, 0) \
  X(52, 2, 2, 8, 8, 0)  \
  X(53, 2, 2, 8, 4, 0)  \
  X(54, 1, 2, 8, 16, 0) \
  X(55, 2, 4, 8, 8, 0)  \
  X(56, 4, 4, 8, 4, 0)  \
  X(57, 4, 4, 8, 8, 0)  \
  X(58, 2, 4, 8, 16, 1) \
  X(59, 2, 4, 8, 16, 0)

constexpr int kFirstLeanRecipe = 40;
constexpr int kEndLeanRecipe = 60;

// LDS row stride (floats) of the wave-pipeline kernel's staged tile: the
// smallest multiple of 4 >= n, up to n + 12, for which lane rows rstep tile
// rows apart start 16 banks apart (of 32), else n
constexpr int wave_row_stride(int n, int rstep) {
  for (int s = n; s <= n + 12; s += 4)
    if ((s * rstep) % 32 == 16) return s;
  return n;
}

// staged floats of one channel in a wave's ring slot: the input tile rounded
// up to 256 floats, plus warea expanded weight floats (64 canonical, 128
// all-ones)
constexpr long wave_slot_floats(int r, int cc, int lw, int s, int d, int warea) {
  const int th = (64 / lw) * r, tw = lw * cc;
  const int tih = (th - 1) * s + 2 * d + 1, tiw = (tw - 1) * s + 2 * d + 1;
  const int lstr = wave_row_stride((tiw + 6) / 4 * 4, r * s);
  return (static_cast<long>(tih) * lstr + 255) / 256 * 256 + warea;
}
// ring slots per wave: fp32 channels are DMA'd into LDS three channels ahead
// (4 slots), or two (3 slots) for stride-1 tilings where 4 would leave a
// compute unit fewer than 8 waves' worth of LDS (160 KB / 8 per wave; timed
// on the 4 x 4 outputs-per-lane tilings); bf16 stages through registers
// (2 slots)
constexpr int wave_nslot(int r, int cc, int lw, int ws, int s, int d, int warea, bool bf16) {
  if (bf16) return 2;
  const long per_wave = (ws >= 8 ? 160L * 1024 / ws : 20L * 1024);
  return s != 1 || 4 * 4 * wave_slot_floats(r, cc, lw, s, d, warea) <= per_wave ? 4 : 3;
}
// LDS floats of one wave-pipeline workgroup: per wave a ring of nslot
// slots, or the partial-sum exchange of 2 slots per wave, whichever is larger
constexpr long wave_lds_floats(int r, int cc, int lw, int ws, int s, int d, int warea, bool bf16) {
  const long ring = wave_nslot(r, cc, lw, ws, s, d, warea, bf16) * wave_slot_floats(r, cc, lw, s, d, warea);
  const long xch = static_cast<long>(ws) * 2 * r * cc * 64;
  return ws * ring > xch ? ws * ring : xch;
}
constexpr int kNumRecipes = 40;

// pipe: the wave-pipeline kernel reads the next channel from LDS into a
// second register set while it computes the current one (fp32, canonical
// library only)
struct RecipeInfo {
  int r, cc, lw, wf, ws, cpw, pipe;
};

#ifndef __HIPCC_RTC__   // host side
// geometry of a recipe, and whether its LDS footprint fits for (stride, dilation)
RecipeInfo recipe_info(int id);
bool recipe_fits(int id, int stride, int dil, bool bf16, int lib);
// recipes compiled for a pattern library (the canonical library gets all)
bool recipe_compiled(int lib, int id);

struct ConvPlan {
  int recipe = 0;
  int ksplit = 1;   // channel split over workgroups (needs scratch, see split_bytes)
};

// bf16 layers as a zero-filled dense contraction on the matrix cores
// (mfma_conv.hip): the plan's recipe id, whether a layer can run so (c_in a
// multiple of 32, no fused max pool, offsets within 32 bits), the scratch it
// needs (the expanded weights and bias) and its launch (p.part = scratch).
constexpr int kRecipeMfma = 64;

// layers with at most four input channels (a network's first layer; fp32 or
// bf16) as dense 3 x 3 taps expanded in LDS (conv_pp_cin.hip): the plan's
// recipe id, whether a layer can run so (stride 1, dilation 1, pad 1, no
// fused epilogue other than ReLU, any pattern library) and its launch
constexpr int kRecipeCin = 60;
bool cin_eligible(const ConvParams& p, bool bf16_act);
hipError_t launch_cin_conv(const ConvParams& p, bool bf16_act, hipStream_t st);

// layers with at most 8 output channels (one slot group: a network's
// image-producing last layer), fp32 or bf16, stride 1, dilation 1, pad 1,
// width a multiple of 4, no fused epilogue other than ReLU, the expanded
// weights within 60 KB of LDS (conv_pp_fewout.hip): dense taps over every
// channel with no dispatch, so the planner takes it for bf16 layers of the
// all-ones library
constexpr int kRecipeFewOut = 61;
bool fewout_eligible(const ConvParams& p);
hipError_t launch_fewout_conv(const ConvParams& p, bool bf16_act, hipStream_t st);
bool mfma_eligible(const ConvParams& p);
size_t mfma_bytes(const ConvParams& p);
bool mfma_long_k(const ConvParams& p);   // k steps of 64 (else 32)
int mfma_groups(const ConvParams& p);    // wave groups per tile splitting its k steps (1 or 2)
hipError_t launch_mfma_conv(const ConvParams& p, hipStream_t st);   // PP_PREPARED in p.flags: no expansion
hipError_t launch_mfma_expand(const ConvParams& p, void* out, hipStream_t st);   // the weights into out

// allow_split: the caller can provide scratch (a channel split's partial
// sums, or the matrix-core form's expanded weights: kRecipeMfma).  With
// PP_MAXPOOL2 in p.flags only plans that can fuse the pool are chosen (a
// split, whose second pass pools, or a tiling with whole windows per lane),
// with PP_ACCUMULATE, PP_PIXSHUF2 or PP_UPSAMPLE2 only wave-pipeline
// tilings, and recipe -1 means none can.  (p.h, p.w are the conv's input
// size: the upsampled size with PP_UPSAMPLE2.)
// no_lean: plan among the wave-pipeline tilings only (the run-time compiled
// kernels of pp_jit_library exist for those)
ConvPlan plan_conv(const ConvParams& p, int lib, bool bf16, bool allow_split, bool no_lean = false);
// scratch bytes a plan needs (its partial-sum blocks, or the matrix-core
// form's expanded weights); 0 for none
size_t split_bytes(const ConvPlan& plan, const ConvParams& p);
hipError_t launch_conv(int lib, const ConvPlan& plan, const ConvParams& p, bool bf16_act, hipStream_t st);

template <int LIB, int S, int D, class TA>
hipError_t launch_recipe(int id, const ConvParams& p, hipStream_t st);

// wave-pipeline kernel, canonical (kLibCanon8) and all-ones (kLibDense9) libraries
template <int LIB, int S, int D, class TA>
hipError_t launch_wave_recipe(int id, const ConvParams& p, hipStream_t st);

// lean kernel (conv_pp_lean.hip)
inline bool is_lean_recipe(int id) { return id >= kFirstLeanRecipe && id < kEndLeanRecipe; }
hipError_t launch_lean_recipe(int id, const ConvParams& p, bool bf16_act, hipStream_t st);
// LDS bytes of a lean tiling for fp32 or bf16 activations at stride 1 and
// dilation (= pad) 1, or fp32 at dilation 2 or stride 2 (0: not compiled
// for that case, or does not fit); whether it stages by 16-byte DMAs (image
// width a multiple of 4 fp32 / 8 bf16 elements)
long lean_lds_bytes(int id, bool bf16 = false, int dil = 1, int stride = 1);
// the tilings also built to read prepared weights (ConvParams::wprep; for
// bf16 activations those of them lean_lds_bytes(id, true) admits)
bool lean_pw_tiling(int id);
// bytes of a layer's prepared lean weights (fp32), and their expansion from
// the blob's fp32 or bf16 weights
size_t lean_prepared_bytes(const ConvParams& p);
hipError_t launch_lean_expand(const ConvParams& p, bool bf16_w, void* out, hipStream_t st);
bool lean_v4(int id);

#endif

}  // namespace pp
