// conv_pp_cin.hip -- pattern/connectivity-pruned 3x3 convolution of a layer
// with at most four input channels (a network's first layer: an RGB or
// one-channel image), fp32 or bf16, stride 1, dilation 1, pad 1, any pattern library.
//
// Same result as the other kernels (pattern + connectivity pruning, Sec. 2;
// compact storage, Sec. 3; conv fused with bias and activation, Sec. 3).
// With so few input channels the channel loop that the other kernels are
// built around has one to four steps, and their per-channel machinery (ring
// staging, slot tests, pattern dispatch) costs more than the arithmetic.  So
// here a workgroup stages its whole input tile (every channel) once, each
// wave expands its slot group's kept kernels into dense 3x3 taps in LDS
// (zeros for pruned kernels and for taps outside a kernel's pattern: at most
// 36 MACs per output, where the dispatch would cost more), and the wave then
// computes its 8 filters one after the other over registers that hold every
// input a lane needs.
//
// Tile: a wave covers 32 x 8 outputs (lanes are 8 across x 8 down, 4
// consecutive outputs of a row each) for half a slot group (4 of its 8
// reordered filters); a workgroup holds kCinWPG such waves over the same
// tile, kCinWPG / 2 slot groups.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "conv_pp.hpp"

namespace pp {
namespace kern {

constexpr int kCinTW = 32, kCinTH = 8;   // output tile
constexpr int kCinWPG = 8;               // waves per workgroup
constexpr int kCinSPW = 4;               // slots (filters) per wave
constexpr int kCinGPG = kCinWPG * kCinSPW / 8;   // slot groups per workgroup
constexpr int kCinLS = 36;               // staged row stride (floats): >= 34, a multiple of 4

// BF: bf16 activations and weights, widened to fp32 on their way into LDS
// (exact), fp32 sums, one rounding at the store.
template <int CIN, bool BF>
__global__ __launch_bounds__(64 * kCinWPG) void pp_conv3x3_cin_kernel(ConvParams a) {
  constexpr int WPS = (CIN * 9 + 3) / 4 * 4;   // expanded taps of one slot, padded to 16 bytes
  constexpr int SR = kCinTH + 2, SC = kCinTW + 2;
  __shared__ __attribute__((aligned(16))) float xs[CIN][SR][kCinLS];
  __shared__ __attribute__((aligned(16))) float ws[kCinWPG][kCinSPW][WPS];
  __shared__ uint32_t perm_s[kCinWPG][kCinSPW];
  __shared__ uint16_t masks_s[kCinWPG][256];
  __shared__ float bias_s[kCinWPG][kCinSPW];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wk = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int gchunks = (a.n_groups + kCinGPG - 1) / kCinGPG;
  uint32_t blk = blockIdx.x;
  const int gc = blk % gchunks;
  blk /= gchunks;
  const int tx = blk % a.tiles_x;
  blk /= a.tiles_x;
  const int ty = blk % a.tiles_y;
  const int img = blk / a.tiles_y;
  const int oy0 = ty * kCinTH, ox0 = tx * kCinTW;

  // ---- the input tile of every channel (pad 1: zeros outside the image);
  // staged column j holds input column ox0 - 1 + j
  const size_t xoff = static_cast<size_t>(img) * CIN * a.h * a.w;
  const float* x = static_cast<const float*>(a.x) + xoff;
  const uint16_t* xb = static_cast<const uint16_t*>(a.x) + xoff;
  {
    // every load first, then every store: one memory round trip
    constexpr int NT = 64 * kCinWPG, NST = (CIN * SR * SC + NT - 1) / NT;
    float v[NST];
#pragma unroll
    for (int k = 0; k < NST; ++k) {
      const int i = tid + NT * k;
      const int c = i / (SR * SC), r = (i / SC) % SR, j = i % SC;
      const int gy = oy0 - 1 + r, gx = ox0 - 1 + j;
      v[k] = 0.0f;
      if (i < CIN * SR * SC && gy >= 0 && gy < a.h && gx >= 0 && gx < a.w) {
        const size_t at = (static_cast<size_t>(c) * a.h + gy) * a.w + gx;
        v[k] = BF ? __uint_as_float(static_cast<uint32_t>(xb[at]) << 16) : x[at];
      }
    }
#pragma unroll
    for (int k = 0; k < NST; ++k) {
      const int i = tid + NT * k;
      if (i < CIN * SR * SC) xs[i / (SR * SC)][(i / SC) % SR][i % SC] = v[k];
    }
  }

  // ---- this wave's slots s0 .. s0 + 3 of slot group g, expanded: lane 4 c +
  // j writes kernel (slot s0 + j, channel c) as 9 dense taps.  Its stored taps start after those of the
  // kept slots before it in the (group, channel) entry.  Every offset read
  // from the blob is clamped to the weights the blob holds.
  const int g = gc * kCinGPG + wk / 2, s0 = (wk & 1) * kCinSPW;
  const bool live = g < a.n_groups;
  const uint32_t np = static_cast<uint32_t>(a.n_patterns);
  if (live) {
    // the pattern library into this wave's LDS copy, loaded alongside the
    // entries below (a wave's LDS writes complete before its later reads)
    const uint16_t* masks = reinterpret_cast<const uint16_t*>(a.blob + a.off_masks);
    for (uint32_t i = lane; i < np && i < 256u; i += 64) masks_s[wk][i] = masks[i];
  }
  if (live && lane < kCinSPW * CIN) {
    const int j = lane % kCinSPW, c = lane / kCinSPW, s = s0 + j;
    const uint32_t e = static_cast<uint32_t>(g) * a.c_in + c;
    // the entry's offset word, its 8 pattern codes and their masks are
    // independent loads (no chain of dependent reads per slot)
    const uint32_t wo = reinterpret_cast<const uint32_t*>(a.blob + a.off_woff)[e];
    const uint2 cw = *reinterpret_cast<const uint2*>(a.blob + a.off_codes + 8u * e);
    const float* wts = reinterpret_cast<const float*>(a.blob + a.off_w);
    const uint16_t* wtb = reinterpret_cast<const uint16_t*>(a.blob + a.off_w);
    const uint32_t last = a.n_wt ? a.n_wt - 1 : 0u;
    uint32_t mk[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const uint32_t code = ((t < 4 ? cw.x : cw.y) >> (8 * (t & 3))) & 0xFFu;
      mk[t] = masks_s[wk][code < np ? code : np - 1];
    }
    const uint32_t kept = wo >> 24;
    uint32_t off = wo & 0xFFFFFFu;
    uint32_t m = 0;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const uint32_t kt = ((kept >> t) & 1u) ? mk[t] : 0u;
      // (bf16 kernels are padded to an even element count)
      if (t < s) off += BF ? (__builtin_popcount(kt) + 1u) & ~1u : __builtin_popcount(kt);
      if (t == s) m = kt;
    }
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      float v = 0.0f;
      if ((m >> t) & 1u) {
        const uint32_t k = min(off + __builtin_popcount(m & ((1u << t) - 1u)), last);
        v = BF ? __uint_as_float(static_cast<uint32_t>(wtb[k]) << 16) : wts[k];
      }
      ws[wk][j][9 * c + t] = v;
    }
    if (c == 0) {
      perm_s[wk][j] = reinterpret_cast<const uint32_t*>(a.blob + a.off_perm)[8 * g + s];
      bias_s[wk][j] = reinterpret_cast<const float*>(a.blob + a.off_bias)[8 * g + s];
#pragma unroll
      for (int t = 9 * CIN; t < WPS; ++t) ws[wk][j][t] = 0.0f;
    }
  }
  __syncthreads();
  if (!live) return;

  // ---- a lane's inputs: rows ly .. ly + 2, staged columns 4 lx .. 4 lx + 5
  const int lx = lane & 7, ly = lane >> 3;
  float p[CIN][3][6];
#pragma unroll
  for (int c = 0; c < CIN; ++c)
#pragma unroll
    for (int r = 0; r < 3; ++r) {
      const float4 u = *reinterpret_cast<const float4*>(&xs[c][ly + r][4 * lx]);
      const float2 v = *reinterpret_cast<const float2*>(&xs[c][ly + r][4 * lx + 4]);
      p[c][r][0] = u.x; p[c][r][1] = u.y; p[c][r][2] = u.z; p[c][r][3] = u.w;
      p[c][r][4] = v.x; p[c][r][5] = v.y;
    }

  const bool relu = (a.flags & PP_RELU) != 0;
  const int oy = oy0 + ly, ox = ox0 + 4 * lx;
  const bool vec = (a.wo % 4 == 0) && ox + 3 < a.wo;
  const size_t yoff = static_cast<size_t>(img) * a.c_out * a.ho * a.wo;
  float* y = static_cast<float*>(a.y) + yoff;
  uint16_t* yb = static_cast<uint16_t*>(a.y) + yoff;
  // the wave's filters one after the other, each slot's taps read from LDS
  // while the slot before it computes
  constexpr int NW4 = WPS / 4;
  float4 wv[NW4];
#pragma unroll
  for (int k = 0; k < NW4; ++k) wv[k] = *reinterpret_cast<const float4*>(&ws[wk][0][4 * k]);
#pragma unroll
  for (int s = 0; s < kCinSPW; ++s) {
    float4 wn[NW4];
    if (s + 1 < kCinSPW) {
#pragma unroll
      for (int k = 0; k < NW4; ++k)
        wn[k] = *reinterpret_cast<const float4*>(&ws[wk][s + 1 < kCinSPW ? s + 1 : 0][4 * k]);
    }
    const float* wf = reinterpret_cast<const float*>(wv);
    float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int c = 0; c < CIN; ++c)
#pragma unroll
      for (int ky = 0; ky < 3; ++ky)
#pragma unroll
        for (int kx = 0; kx < 3; ++kx) {
          const float w = wf[9 * c + 3 * ky + kx];
#pragma unroll
          for (int q = 0; q < 4; ++q) acc[q] = __builtin_fmaf(w, p[c][ky][kx + q], acc[q]);
        }
    const uint32_t o = __builtin_amdgcn_readfirstlane(perm_s[wk][s]);
    if (o < static_cast<uint32_t>(a.c_out) && oy < a.ho) {   // (o >= c_out: a padding slot)
      const float b = bias_s[wk][s];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[q] += b;
        if (relu) acc[q] = fmaxf(acc[q], 0.0f);
      }
      const size_t ro = (static_cast<size_t>(o) * a.ho + oy) * a.wo;
      if constexpr (BF) {
        // round to nearest even (finite values)
        uint32_t u[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          u[q] = __float_as_uint(acc[q]);
          u[q] = (u[q] + 0x7FFFu + ((u[q] >> 16) & 1u)) >> 16;
        }
        uint16_t* row = yb + ro;
        if (vec) {
          *reinterpret_cast<uint2*>(row + ox) = make_uint2(u[0] | (u[1] << 16), u[2] | (u[3] << 16));
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (ox + q < a.wo) row[ox + q] = static_cast<uint16_t>(u[q]);
        }
      } else {
        float* row = y + ro;
        if (vec) {
          *reinterpret_cast<float4*>(row + ox) = make_float4(acc[0], acc[1], acc[2], acc[3]);
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (ox + q < a.wo) row[ox + q] = acc[q];
        }
      }
    }
    if (s + 1 < kCinSPW) {
#pragma unroll
      for (int k = 0; k < NW4; ++k) wv[k] = wn[k];
    }
  }
}

}  // namespace kern

bool cin_eligible(const ConvParams& p, bool bf16_act) {
  (void)bf16_act;
  return p.c_in >= 1 && p.c_in <= 4 && p.stride == 1 && p.dil == 1 && p.pad == 1 && p.ho == p.h &&
         p.wo == p.w && (p.flags & (PP_MAXPOOL2 | PP_ACCUMULATE | PP_PIXSHUF2 | PP_UPSAMPLE2)) == 0;
}

hipError_t launch_cin_conv(const ConvParams& p0, bool bf16, hipStream_t st) {
  if (!cin_eligible(p0, bf16) || p0.n < 1 || p0.n_groups < 1) return hipErrorInvalidConfiguration;
  ConvParams p = p0;
  p.tiles_x = (p.wo + kern::kCinTW - 1) / kern::kCinTW;
  p.tiles_y = (p.ho + kern::kCinTH - 1) / kern::kCinTH;
  const long gchunks = (p.n_groups + kern::kCinGPG - 1) / kern::kCinGPG;
  const long nb = static_cast<long>(p.n) * p.tiles_y * p.tiles_x * gchunks;
  if (nb < 1 || nb > 0x7FFFFFFFL) return hipErrorInvalidConfiguration;
  const dim3 grid(static_cast<uint32_t>(nb)), block(64 * kern::kCinWPG);
#define PP_CIN(C)                                                                               \
  if (bf16) hipLaunchKernelGGL((kern::pp_conv3x3_cin_kernel<C, true>), grid, block, 0, st, p);  \
  else hipLaunchKernelGGL((kern::pp_conv3x3_cin_kernel<C, false>), grid, block, 0, st, p);
  switch (p.c_in) {
    case 1: PP_CIN(1) break;
    case 2: PP_CIN(2) break;
    case 3: PP_CIN(3) break;
    default: PP_CIN(4) break;
  }
#undef PP_CIN
  return hipGetLastError();
}

}  // namespace pp
