// conv_pp_fewout.hip -- pruned 3x3 convolution of a layer with at most 8
// output channels (a network's image-producing last layer, e.g. 64 -> 3),
// fp32 or bf16 activations, stride 1, dilation 1, pad 1, any pattern library.
//
// Same result as the other kernels (pattern + connectivity pruning, Sec. 2;
// compact storage, Sec. 3; conv fused with bias and activation, Sec. 3).
// A layer with one slot group gives the other kernels one 8-slot dispatch
// per channel step for at most 8 x 9 taps of work, on the largest maps of a
// network (the output image), so that per-channel machinery dominates.  Here
// the workgroup first expands the whole layer's kept kernels into dense 3x3
// taps in LDS (a few KB: zeros for pruned kernels and off-pattern taps, so
// a pruned layer does dense work -- the planner takes this kernel for the
// all-ones library), and each wave then walks the input channels with no
// dispatch at all: per channel it loads its lanes' input rows straight from
// global memory one channel ahead (each input element reaches the chip
// once; halo overlap between neighbouring lanes hits the caches) and does
// NF x 9 taps x 8 outputs of FMAs per lane, weights read from LDS.
//
// Tile: a wave covers 64 x 8 outputs (16 lanes across x 4 down, a 2 x 4
// block per lane); a workgroup is 4 waves stacked vertically (64 x 32).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "conv_pp.hpp"

namespace pp {
namespace kern {

constexpr int kFewTW = 64, kFewTH = 32;   // workgroup tile (4 waves of 64 x 8)
constexpr int kFewLds = 60 * 1024;        // bytes of the expanded weight table at most

template <int NF>
struct FewGeo {
  static constexpr int WPC = (NF * 9 + 3) / 4 * 4;   // expanded taps of one channel (all NF slots)
};

__device__ __forceinline__ uint32_t few_bf16(float f) {   // round to nearest even (finite values)
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

template <int NF, class TA>
__global__ __launch_bounds__(256) void pp_conv3x3_fewout_kernel(ConvParams a) {
  constexpr int WPC = FewGeo<NF>::WPC;
  constexpr bool BF = sizeof(TA) == 2;
  extern __shared__ __attribute__((aligned(16))) float wtab[];   // [c_in][WPC]
  __shared__ uint16_t masks_s[256];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wk = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tiles_x = a.tiles_x, tiles_y = a.tiles_y;
  int blk = blockIdx.x;
  const int tx = blk % tiles_x;
  blk /= tiles_x;
  const int ty = blk % tiles_y;
  const int img = blk / tiles_y;

  // ---- the layer's kept kernels as dense taps: entry (c, s) at c * WPC + 9 s.
  // Its stored taps start after those of the kept slots before it in the
  // (group 0, channel c) entry; every offset read from the blob is clamped to
  // the weights the blob holds.
  const uint32_t np = static_cast<uint32_t>(a.n_patterns);
  {
    const uint16_t* masks = reinterpret_cast<const uint16_t*>(a.blob + a.off_masks);
    for (uint32_t i = tid; i < np && i < 256u; i += 256) masks_s[i] = masks[i];
  }
  __syncthreads();
  const uint32_t last = a.n_wt ? a.n_wt - 1 : 0u;
  for (int e = tid; e < a.c_in * NF; e += 256) {
    const int c = e / NF, s = e % NF;
    const uint32_t wo = reinterpret_cast<const uint32_t*>(a.blob + a.off_woff)[c];
    const uint2 cw = *reinterpret_cast<const uint2*>(a.blob + a.off_codes + 8u * c);
    const uint32_t kept = wo >> 24;
    uint32_t off = wo & 0xFFFFFFu, m = 0;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const uint32_t code = ((t < 4 ? cw.x : cw.y) >> (8 * (t & 3))) & 0xFFu;
      const uint32_t kt = ((kept >> t) & 1u) ? masks_s[code < np ? code : np - 1] : 0u;
      const uint32_t n = __builtin_popcount(kt);
      if (t < s) off += BF ? n + (n & 1u) : n;
      if (t == s) m = kt;
    }
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      float v = 0.0f;
      if ((m >> t) & 1u) {
        const uint32_t k = min(off + __builtin_popcount(m & ((1u << t) - 1u)), last);
        v = BF ? __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(a.blob + a.off_w)[k]) << 16)
               : reinterpret_cast<const float*>(a.blob + a.off_w)[k];
      }
      wtab[c * WPC + 9 * s + t] = v;
    }
    if (s == 0)
      for (int t = 9 * NF; t < WPC; ++t) wtab[c * WPC + t] = 0.0f;
  }
  __syncthreads();

  // ---- this lane's 2 x 4 outputs and the 4 x 6 inputs they read per channel
  const int lx = lane & 15, ly = lane >> 4;
  const int oy = ty * kFewTH + wk * 8 + 2 * ly;   // first of the lane's 2 output rows
  const int ox = tx * kFewTW + 4 * lx;            // first of its 4 columns (w is a multiple of 4)
  const bool lane_in = ox < a.w;
  const size_t cstride = static_cast<size_t>(a.h) * a.w;
  // raw-buffer loads through a per-channel descriptor: an offset outside the
  // channel (rows above or below the image, the column left of the first or
  // right of the last one, lanes past the width) reads zero -- the padding --
  // with no branch and no select.  The byte offsets are the same for every
  // channel.
  constexpr uint32_t kOut = 0x80000000u;
  constexpr uint32_t ES = sizeof(TA);
  uint32_t om[4], ol[4], orr[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int gy = oy - 1 + r;
    const bool rv = lane_in && gy >= 0 && gy < a.h;
    const uint32_t base = static_cast<uint32_t>(gy * a.w + ox) * ES;
    om[r] = rv ? base : kOut;
    ol[r] = rv && ox > 0 ? base - ES : kOut;
    orr[r] = rv && ox + 4 < a.w ? base + 4 * ES : kOut;
  }
  const TA* x = static_cast<const TA*>(a.x) + static_cast<size_t>(img) * a.c_in * cstride;
  const int chan_bytes = static_cast<int>(cstride * ES);
  auto load_patch = [&](int c, float (&pt)[4][6]) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<TA*>(x + static_cast<size_t>(c) * cstride), static_cast<short>(0), chan_bytes, 0x00020000);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      if constexpr (BF) {
        const uint2 u = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(xr, om[r], 0, 0));
        pt[r][1] = __uint_as_float(u.x << 16); pt[r][2] = __uint_as_float(u.x & 0xFFFF0000u);
        pt[r][3] = __uint_as_float(u.y << 16); pt[r][4] = __uint_as_float(u.y & 0xFFFF0000u);
        pt[r][0] = __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(xr, ol[r], 0, 0)) << 16);
        pt[r][5] = __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(xr, orr[r], 0, 0)) << 16);
      } else {
        const float4 u = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(xr, om[r], 0, 0));
        pt[r][1] = u.x; pt[r][2] = u.y; pt[r][3] = u.z; pt[r][4] = u.w;
        pt[r][0] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xr, ol[r], 0, 0));
        pt[r][5] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xr, orr[r], 0, 0));
      }
    }
  };

  float acc[NF][2][4];
#pragma unroll
  for (int s = 0; s < NF; ++s)
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[s][r][q] = 0.0f;

  // one channel: FMAs over pt while the next channel's rows load into nx
  // (unconditionally: the last step reloads its own channel, so the loads
  // are not in a branch the compiler would place after the FMAs)
  auto step = [&](int c, float (&pt)[4][6], float (&nx)[4][6]) __attribute__((always_inline)) {
    load_patch(c + 1 < a.c_in ? c + 1 : c, nx);
    const float* wc = wtab + c * WPC;
#pragma unroll
    for (int s = 0; s < NF; ++s)
#pragma unroll
      for (int ky = 0; ky < 3; ++ky)
#pragma unroll
        for (int kx = 0; kx < 3; ++kx) {
          const float wv = wc[9 * s + 3 * ky + kx];
#pragma unroll
          for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[s][r][q] = __builtin_fmaf(wv, pt[r + ky][q + kx], acc[s][r][q]);
        }
  };
  float pa[4][6], pb[4][6];
  load_patch(0, pa);
#pragma unroll 1
  for (int c = 0; c < a.c_in; c += 2) {
    step(c, pa, pb);
    if (c + 1 < a.c_in) step(c + 1, pb, pa);
  }

  // ---- epilogue: + bias, ReLU, store through perm (slot s of group 0)
  if (!lane_in) return;
  const bool relu = (a.flags & PP_RELU) != 0;
  const uint32_t* perm = reinterpret_cast<const uint32_t*>(a.blob + a.off_perm);
  const float* biasv = reinterpret_cast<const float*>(a.blob + a.off_bias);
  TA* y = static_cast<TA*>(a.y) + static_cast<size_t>(img) * a.c_out * cstride;
#pragma unroll
  for (int s = 0; s < NF; ++s) {
    const uint32_t o = perm[s];
    if (o >= static_cast<uint32_t>(a.c_out)) continue;   // padding slot
    const float b = biasv[s];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      if (oy + r >= a.h) continue;
      float v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[q] = acc[s][r][q] + b;
        if (relu) v[q] = fmaxf(v[q], 0.0f);
      }
      TA* row = y + static_cast<size_t>(o) * cstride + static_cast<size_t>(oy + r) * a.w + ox;
      if constexpr (BF) {
        *reinterpret_cast<uint2*>(row) =
            make_uint2(few_bf16(v[0]) | (few_bf16(v[1]) << 16), few_bf16(v[2]) | (few_bf16(v[3]) << 16));
      } else {
        *reinterpret_cast<float4*>(row) = make_float4(v[0], v[1], v[2], v[3]);
      }
    }
  }
}

template <int NF, class TA>
hipError_t launch_fewout(const ConvParams& p, size_t lds, hipStream_t st) {
  const dim3 grid(static_cast<uint32_t>(static_cast<long>(p.n) * p.tiles_y * p.tiles_x)), block(256);
  hipLaunchKernelGGL((pp_conv3x3_fewout_kernel<NF, TA>), grid, block, lds, st, p);
  return hipGetLastError();
}

}  // namespace kern

static int fewout_nf(int c_out) { return c_out <= 3 ? 3 : c_out <= 4 ? 4 : 8; }

static size_t fewout_lds(const ConvParams& p) {
  const int nf = fewout_nf(p.c_out);
  const size_t wpc = nf == 3 ? kern::FewGeo<3>::WPC : nf == 4 ? kern::FewGeo<4>::WPC : kern::FewGeo<8>::WPC;
  return static_cast<size_t>(p.c_in) * wpc * sizeof(float);
}

bool fewout_eligible(const ConvParams& p) {
  return p.n_groups == 1 && p.c_out >= 1 && p.c_out <= 8 && p.c_in >= 1 && p.stride == 1 && p.dil == 1 &&
         p.pad == 1 && p.ho == p.h && p.wo == p.w && p.w % 4 == 0 &&
         static_cast<size_t>(p.h) * p.w * sizeof(float) < 0x80000000ull &&   // one channel within a buffer range
         (p.flags & (PP_MAXPOOL2 | PP_ACCUMULATE | PP_PIXSHUF2 | PP_UPSAMPLE2)) == 0 &&
         fewout_lds(p) <= static_cast<size_t>(kern::kFewLds);
}

hipError_t launch_fewout_conv(const ConvParams& p0, bool bf16_act, hipStream_t st) {
  if (!fewout_eligible(p0) || p0.n < 1) return hipErrorInvalidConfiguration;
  ConvParams p = p0;
  p.tiles_x = (p.w + kern::kFewTW - 1) / kern::kFewTW;
  p.tiles_y = (p.h + kern::kFewTH - 1) / kern::kFewTH;
  const long nb = static_cast<long>(p.n) * p.tiles_y * p.tiles_x;
  if (nb < 1 || nb > 0x7FFFFFFFL) return hipErrorInvalidConfiguration;
  const size_t lds = fewout_lds(p);
  switch (fewout_nf(p.c_out)) {
    case 3: return bf16_act ? kern::launch_fewout<3, uint16_t>(p, lds, st) : kern::launch_fewout<3, float>(p, lds, st);
    case 4: return bf16_act ? kern::launch_fewout<4, uint16_t>(p, lds, st) : kern::launch_fewout<4, float>(p, lds, st);
    default: return bf16_act ? kern::launch_fewout<8, uint16_t>(p, lds, st) : kern::launch_fewout<8, float>(p, lds, st);
  }
}

}  // namespace pp
