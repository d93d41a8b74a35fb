// conv_pp.hip -- pattern/connectivity-pruned 3x3 convolution for gfx950.
//
// One launch computes y = act(conv(x, W_pruned) + b) for a PPK1-packed layer
// (pattern + connectivity pruning, Sec. 2; compact storage and filter
// reorder, Sec. 3; conv fused with bias and activation, Sec. 3).
//
// Mapping to CDNA4:
//   * A workgroup owns one spatial output tile of one image and WF*NG slot
//     groups (8 packed filters each).  Its input halo tile is staged from HBM
//     into LDS one chunk of CCH input channels at a time (coalesced along
//     rows, zero-filled outside the image) and shared by every filter of the
//     workgroup.
//   * Lanes are output pixels: each lane owns an R x CC block of outputs for
//     all 8*NG filters of its wave, so the whole 3x3 neighbourhood it needs
//     for one input channel ("patch") is read from LDS once and reused by
//     every kept kernel of that channel.
//   * Everything that depends on the sparsity structure is wave-uniform: the
//     per-(group, channel) code word, the weight offset and the weights are
//     scalar loads into SGPRs, and the pattern selects a code path through a
//     uniform branch whose tap offsets are compile-time constants.  No lane
//     ever diverges on the pruning structure.
//   * WS waves of a workgroup may split the channels of each chunk; their
//     partial sums are reduced through LDS in a fixed order at the end, so
//     results are deterministic.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "conv_pp.hpp"

namespace pp {
namespace {

// ---------------------------------------------------------------------------
// scalar (wave-uniform) loads from the read-only blob
// ---------------------------------------------------------------------------
template <class T>
__device__ __forceinline__ T sload(const uint8_t* base, uint32_t byte_off) {
  // 32-bit pieces through the constant address space: uniform addresses
  // become s_load_dword{,x2,x4} into SGPRs
  typedef const __attribute__((address_space(4))) uint32_t* cptr;
  static_assert(sizeof(T) % 4 == 0, "scalar loads move whole dwords");
  const cptr src = (cptr)(base + byte_off);
  union {
    T v;
    uint32_t u[sizeof(T) / 4];
  } r;
#pragma unroll
  for (int i = 0; i < static_cast<int>(sizeof(T) / 4); ++i) r.u[i] = src[i];
  return r.v;
}

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

__device__ __forceinline__ float load_act(const float* p, size_t i) { return p[i]; }
__device__ __forceinline__ float load_act(const uint16_t* p, size_t i) {
  return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
}
__device__ __forceinline__ void store_act(float* p, size_t i, float v) { p[i] = v; }
__device__ __forceinline__ void store_act(uint16_t* p, size_t i, float v) {
  uint32_t u = __float_as_uint(v);
  u += 0x7FFFu + ((u >> 16) & 1u);   // round to nearest even (finite values)
  p[i] = static_cast<uint16_t>(u >> 16);
}

// canonical 8-pattern library (4 taps each, all containing the centre)
constexpr uint32_t kCanon8[8] = {0x03A, 0x0B2, 0x0B8, 0x09A, 0x01B, 0x036, 0x0D8, 0x1B0};

constexpr int nth_tap(uint32_t mask, int n) {
  for (int t = 0; t < 9; ++t)
    if ((mask >> t) & 1u) {
      if (n == 0) return t;
      --n;
    }
  return -1;
}

// acc[r][q] += w * x(r*S + ky*D, q*S + kx*D) for one tap
template <int TAP, int S, int D, int R, int CC, int PR, int PC>
__device__ __forceinline__ void fma_tap(float (&acc)[R][CC], const float (&pt)[PR][PC], float w) {
  constexpr int ky = TAP / 3, kx = TAP % 3;
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int q = 0; q < CC; ++q) acc[r][q] = __builtin_fmaf(w, pt[r * S + ky * D][q * S + kx * D], acc[r][q]);
}

// one 4-tap kernel of compile-time pattern MASK, weights w0..w3 in tap order
template <uint32_t MASK, int S, int D, int R, int CC, int PR, int PC>
__device__ __forceinline__ void apply4(float (&acc)[R][CC], const float (&pt)[PR][PC], float w0, float w1,
                                       float w2, float w3) {
  fma_tap<nth_tap(MASK, 0), S, D>(acc, pt, w0);
  fma_tap<nth_tap(MASK, 1), S, D>(acc, pt, w1);
  fma_tap<nth_tap(MASK, 2), S, D>(acc, pt, w2);
  fma_tap<nth_tap(MASK, 3), S, D>(acc, pt, w3);
}

template <int S, int D, int R, int CC, int PR, int PC>
__device__ __forceinline__ void apply_canon8(uint32_t p, float (&acc)[R][CC], const float (&pt)[PR][PC],
                                             float w0, float w1, float w2, float w3) {
  switch (p) {
    case 0: apply4<kCanon8[0], S, D>(acc, pt, w0, w1, w2, w3); break;
    case 1: apply4<kCanon8[1], S, D>(acc, pt, w0, w1, w2, w3); break;
    case 2: apply4<kCanon8[2], S, D>(acc, pt, w0, w1, w2, w3); break;
    case 3: apply4<kCanon8[3], S, D>(acc, pt, w0, w1, w2, w3); break;
    case 4: apply4<kCanon8[4], S, D>(acc, pt, w0, w1, w2, w3); break;
    case 5: apply4<kCanon8[5], S, D>(acc, pt, w0, w1, w2, w3); break;
    case 6: apply4<kCanon8[6], S, D>(acc, pt, w0, w1, w2, w3); break;
    case 7: apply4<kCanon8[7], S, D>(acc, pt, w0, w1, w2, w3); break;
    default: break;
  }
}

// generic library: taps tested one by one against the runtime mask
template <int S, int D, int R, int CC, int PR, int PC>
__device__ __forceinline__ void apply_generic(uint32_t mask, float (&acc)[R][CC], const float (&pt)[PR][PC],
                                              const uint8_t* blob, uint32_t off_w, uint32_t k, uint32_t n_wt,
                                              bool bf16w) {
  uint32_t q = 0;
  const uint32_t last = n_wt ? n_wt - 1 : 0u;   // clamp: never read past the weights
#define PP_TAP(T)                                                                              \
  if (mask & (1u << T)) {                                                                      \
    const uint32_t kq = min(k + q, last);                                                      \
    float wv;                                                                                  \
    if (bf16w) {                                                                               \
      uint32_t u = sload<uint32_t>(blob, (off_w + 2 * kq) & ~3u);                              \
      wv = (kq & 1) ? bf16_hi(u) : bf16_lo(u);                                                 \
    } else {                                                                                   \
      wv = sload<float>(blob, off_w + 4 * kq);                                                 \
    }                                                                                          \
    fma_tap<T, S, D>(acc, pt, wv);                                                             \
    ++q;                                                                                       \
  }
  PP_TAP(0) PP_TAP(1) PP_TAP(2) PP_TAP(3) PP_TAP(4) PP_TAP(5) PP_TAP(6) PP_TAP(7) PP_TAP(8)
#undef PP_TAP
}

template <int S, int D, int R, int CC, int PR, int PC>
__device__ __forceinline__ void apply_dense9(float (&acc)[R][CC], const float (&pt)[PR][PC], const float* w) {
  fma_tap<0, S, D>(acc, pt, w[0]);
  fma_tap<1, S, D>(acc, pt, w[1]);
  fma_tap<2, S, D>(acc, pt, w[2]);
  fma_tap<3, S, D>(acc, pt, w[3]);
  fma_tap<4, S, D>(acc, pt, w[4]);
  fma_tap<5, S, D>(acc, pt, w[5]);
  fma_tap<6, S, D>(acc, pt, w[6]);
  fma_tap<7, S, D>(acc, pt, w[7]);
  fma_tap<8, S, D>(acc, pt, w[8]);
}

// blockIdx -> logical block so that consecutive logical blocks (which share
// the same input tile) land on the same XCD: the dispatcher sends block b to
// XCD b % 8, and each XCD has its own L2.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t b, uint32_t nb) {
  const uint32_t x = b & 7u, local = b >> 3;
  const uint32_t q0 = nb >> 3, r = nb & 7u, q1 = q0 + (r ? 1u : 0u);
  return x < r ? x * q1 + local : r * q1 + (x - r) * q0 + local;
}

}  // namespace

template <int LIB, int S, int D, int R, int CC, int LW, int NG, int WF, int WS, int CCH, class TA>
__global__ __launch_bounds__(WF* WS * 64) void pp_conv3x3_kernel(ConvParams a) {
  constexpr int LH = 64 / LW;
  constexpr int TH = LH * R, TW = LW * CC;                        // output tile
  constexpr int PR = (R - 1) * S + 2 * D + 1;                     // patch rows
  constexpr int PC = (CC - 1) * S + 2 * D + 1;                    // patch cols
  constexpr int TIH = (TH - 1) * S + 2 * D + 1;                   // input tile rows
  constexpr int TIW = (TW - 1) * S + 2 * D + 1;                   // input tile cols
  constexpr int LSTR = (TIW + 3) / 4 * 4;                         // LDS row stride (floats)
  constexpr int CHSTR = TIH * LSTR;                               // LDS channel stride
  constexpr int NT = WF * WS * 64;
  constexpr int CPW = CCH / WS;                                   // channels per wave per chunk
  constexpr int NACC = NG * 8 * R * CC;
  constexpr int STAGE = CCH * CHSTR;
  constexpr int RED = (WS > 1) ? (WS - 1) * WF * NACC * 64 : 0;
  constexpr int LDS_FLOATS = STAGE > RED ? STAGE : RED;
  constexpr int VW = ((CC * S) % 4 == 0) ? 4 : (((CC * S) % 2 == 0) ? 2 : 1);   // patch read width
  constexpr bool WBF = sizeof(TA) == 2;                           // bf16 weights with bf16 activations
  constexpr int N4 = (VW == 4) ? PC / 4 : 0;                      // patch row: float4 reads,
  constexpr int N2 = (VW >= 2) ? (PC - 4 * N4) / 2 : 0;           // then float2,
  constexpr int N1 = PC - 4 * N4 - 2 * N2;                        // then single floats
  constexpr int STAGE_N = CCH * TIH * TIW;                        // staged elements per chunk
  constexpr int NST = (STAGE_N + NT - 1) / NT;                    // ... per thread
  static_assert(LW * LH == 64, "64 lanes per wave");
  static_assert(CCH % WS == 0, "chunk must split evenly across waves");
  static_assert(LDS_FLOATS * 4 <= 64 * 1024, "LDS budget");

  __shared__ __attribute__((aligned(16))) float lds[LDS_FLOATS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wf = wid % WF, wk = wid / WF;
  const int lx = lane % LW, ly = lane / LW;

  uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
  const int ft = blk % a.n_ftiles;
  blk /= a.n_ftiles;
  const int tx = blk % a.tiles_x;
  blk /= a.tiles_x;
  const int ty = blk % a.tiles_y;
  const int img = blk / a.tiles_y;

  const int oy0 = ty * TH, ox0 = tx * TW;
  const int iy0 = oy0 * S - a.pad, ix0 = ox0 * S - a.pad;
  const int g0 = (ft * WF + wf) * NG;

  const TA* __restrict__ x = static_cast<const TA*>(a.x) + static_cast<size_t>(img) * a.c_in * a.h * a.w;
  const uint8_t* blob = a.blob;

  float acc[NG][8][R][CC];
#pragma unroll
  for (int g = 0; g < NG; ++g)
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int q = 0; q < CC; ++q) acc[g][s][r][q] = 0.0f;

  const int lane_off = (ly * R * S) * LSTR + lx * CC * S;

  for (int cb = 0; cb < a.c_in; cb += CCH) {
    __syncthreads();
    // ---- stage input channels [cb, cb+CCH) of the halo tile into LDS:
    // all loads of this thread first, then all LDS writes
    {
      float v[NST];
#pragma unroll
      for (int k = 0; k < NST; ++k) {
        const int idx = tid + k * NT;
        const int j = idx % TIW;
        const int t2 = idx / TIW;
        const int i = t2 % TIH;
        const int ch = t2 / TIH;
        const int c = cb + ch, gy = iy0 + i, gx = ix0 + j;
        v[k] = 0.0f;
        if (idx < STAGE_N && c < a.c_in && gy >= 0 && gy < a.h && gx >= 0 && gx < a.w)
          v[k] = load_act(x, (static_cast<size_t>(c) * a.h + gy) * a.w + gx);
      }
#pragma unroll
      for (int k = 0; k < NST; ++k) {
        const int idx = tid + k * NT;
        if (idx < STAGE_N) {
          const int j = idx % TIW;
          const int t2 = idx / TIW;
          lds[(t2 / TIH) * CHSTR + (t2 % TIH) * LSTR + j] = v[k];
        }
      }
    }
    __syncthreads();

    const int cl_end = min(CCH, a.c_in - cb);
    for (int cl = wk * CPW; cl < (wk + 1) * CPW && cl < cl_end; ++cl) {
      const int c = cb + cl;
      // ---- patch: the lane's input neighbourhood for channel c
      float pt[PR][PC];
      const float* src = lds + cl * CHSTR + lane_off;
#pragma unroll
      for (int r = 0; r < PR; ++r) {
        const float* row = src + r * LSTR;
#pragma unroll
        for (int i = 0; i < N4; ++i) {
          const float4 v = *reinterpret_cast<const float4*>(row + 4 * i);
          pt[r][4 * i] = v.x; pt[r][4 * i + 1] = v.y; pt[r][4 * i + 2] = v.z; pt[r][4 * i + 3] = v.w;
        }
#pragma unroll
        for (int i = 0; i < N2; ++i) {
          const float2 v = *reinterpret_cast<const float2*>(row + 4 * N4 + 2 * i);
          pt[r][4 * N4 + 2 * i] = v.x; pt[r][4 * N4 + 2 * i + 1] = v.y;
        }
#pragma unroll
        for (int i = 0; i < N1; ++i) pt[r][4 * N4 + 2 * N2 + i] = row[4 * N4 + 2 * N2 + i];
      }
      // ---- every kept kernel of the wave's filters for channel c
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const int grp = g0 + g;
        if (grp >= a.n_groups) continue;
        const uint32_t e = static_cast<uint32_t>(grp) * a.c_in + c;
        const uint2 code = sload<uint2>(blob, a.off_codes + 8 * e);
        const uint32_t wo = sload<uint32_t>(blob, a.off_woff + 4 * e);
        if (LIB == kLibCanon8) {
          if (WBF) {
            uint2 wv[8];
            uint32_t k = min(wo, a.n_wt);
#pragma unroll
            for (int s = 0; s < 8; ++s) {
              const uint32_t p = ((s < 4 ? code.x : code.y) >> (8 * (s & 3))) & 0xFFu;
              wv[s] = sload<uint2>(blob, a.off_w + 2 * min(k, a.n_wt));
              k += (p != 0xFFu) ? 4u : 0u;
            }
#pragma unroll
            for (int s = 0; s < 8; ++s) {
              const uint32_t p = ((s < 4 ? code.x : code.y) >> (8 * (s & 3))) & 0xFFu;
              apply_canon8<S, D>(p, acc[g][s], pt, bf16_lo(wv[s].x), bf16_hi(wv[s].x), bf16_lo(wv[s].y),
                                 bf16_hi(wv[s].y));
            }
          } else {
            float4 wv[8];
            uint32_t k = min(wo, a.n_wt);
#pragma unroll
            for (int s = 0; s < 8; ++s) {
              const uint32_t p = ((s < 4 ? code.x : code.y) >> (8 * (s & 3))) & 0xFFu;
              wv[s] = sload<float4>(blob, a.off_w + 4 * min(k, a.n_wt));
              k += (p != 0xFFu) ? 4u : 0u;
            }
#pragma unroll
            for (int s = 0; s < 8; ++s) {
              const uint32_t p = ((s < 4 ? code.x : code.y) >> (8 * (s & 3))) & 0xFFu;
              apply_canon8<S, D>(p, acc[g][s], pt, wv[s].x, wv[s].y, wv[s].z, wv[s].w);
            }
          }
        } else if (LIB == kLibDense9) {
          uint32_t k = wo;
#pragma unroll
          for (int s = 0; s < 8; ++s) {
            const uint32_t p = ((s < 4 ? code.x : code.y) >> (8 * (s & 3))) & 0xFFu;
            if (p == 0xFFu) continue;
            float w9[9];
            if (WBF) {
              const uint32_t kc = min(k, a.n_wt >= 10 ? a.n_wt - 10 : 0u);
              const uint4 u = sload<uint4>(blob, a.off_w + 2 * kc);
              const uint32_t u4 = sload<uint32_t>(blob, a.off_w + 2 * kc + 16);
              w9[0] = bf16_lo(u.x); w9[1] = bf16_hi(u.x); w9[2] = bf16_lo(u.y); w9[3] = bf16_hi(u.y);
              w9[4] = bf16_lo(u.z); w9[5] = bf16_hi(u.z); w9[6] = bf16_lo(u.w); w9[7] = bf16_hi(u.w);
              w9[8] = bf16_lo(u4);
              k += 10;
            } else {
              const uint32_t kc = min(k, a.n_wt >= 9 ? a.n_wt - 9 : 0u);
              const float4 u = sload<float4>(blob, a.off_w + 4 * kc);
              const float4 v = sload<float4>(blob, a.off_w + 4 * kc + 16);
              const float z = sload<float>(blob, a.off_w + 4 * kc + 32);
              w9[0] = u.x; w9[1] = u.y; w9[2] = u.z; w9[3] = u.w;
              w9[4] = v.x; w9[5] = v.y; w9[6] = v.z; w9[7] = v.w; w9[8] = z;
              k += 9;
            }
            apply_dense9<S, D>(acc[g][s], pt, w9);
          }
        } else {
          uint32_t k = wo;
#pragma unroll
          for (int s = 0; s < 8; ++s) {
            const uint32_t p = ((s < 4 ? code.x : code.y) >> (8 * (s & 3))) & 0xFFu;
            if (p == 0xFFu) continue;
            const uint32_t pc = min(p, static_cast<uint32_t>(a.n_patterns - 1));
            const uint32_t mw = sload<uint32_t>(blob, (a.off_masks + 2 * pc) & ~3u);
            const uint32_t mask = ((pc & 1u) ? (mw >> 16) : mw) & 0x1FFu;
            apply_generic<S, D>(mask, acc[g][s], pt, blob, a.off_w, k, a.n_wt, WBF);
            const uint32_t nt = __builtin_popcount(mask);
            k += WBF ? ((nt + 1u) & ~1u) : nt;
          }
        }
      }
    }
  }

  // ---- reduce the WS channel-split partial sums (fixed order)
  if (WS > 1) {
    __syncthreads();
    float* red = lds;
    if (wk > 0) {
      float* dst = red + static_cast<size_t>((wk - 1) * WF + wf) * NACC * 64 + lane;
      int i = 0;
#pragma unroll
      for (int g = 0; g < NG; ++g)
#pragma unroll
        for (int s = 0; s < 8; ++s)
#pragma unroll
          for (int r = 0; r < R; ++r)
#pragma unroll
            for (int q = 0; q < CC; ++q, ++i) dst[i * 64] = acc[g][s][r][q];
    }
    __syncthreads();
    if (wk > 0) return;
    for (int kk = 1; kk < WS; ++kk) {
      const float* srcp = red + static_cast<size_t>((kk - 1) * WF + wf) * NACC * 64 + lane;
      int i = 0;
#pragma unroll
      for (int g = 0; g < NG; ++g)
#pragma unroll
        for (int s = 0; s < 8; ++s)
#pragma unroll
          for (int r = 0; r < R; ++r)
#pragma unroll
            for (int q = 0; q < CC; ++q, ++i) acc[g][s][r][q] += srcp[i * 64];
    }
  }

  // ---- epilogue: + bias, activation, store to the original channel order
  TA* __restrict__ y = static_cast<TA*>(a.y) + static_cast<size_t>(img) * a.c_out * a.ho * a.wo;
  const bool relu = (a.flags & PP_RELU) != 0;
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int grp = g0 + g;
    if (grp >= a.n_groups) continue;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const uint32_t slot = static_cast<uint32_t>(grp) * 8 + s;
      const uint32_t o = sload<uint32_t>(blob, a.off_perm + 4 * slot);
      if (o >= static_cast<uint32_t>(a.c_out)) continue;   // padding slot
      const float bias = sload<float>(blob, a.off_bias + 4 * slot);
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int oy = oy0 + ly * R + r;
        if (oy >= a.ho) continue;
#pragma unroll
        for (int q = 0; q < CC; ++q) {
          const int ox = ox0 + lx * CC + q;
          if (ox >= a.wo) continue;
          float v = acc[g][s][r][q] + bias;
          if (relu) v = fmaxf(v, 0.0f);
          store_act(y, (static_cast<size_t>(o) * a.ho + oy) * a.wo + ox, v);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// host side: instantiation table and launch
// ---------------------------------------------------------------------------
namespace {

template <int LIB, int S, int D, int R, int CC, int LW, int NG, int WF, int WS, int CCH, class TA>
hipError_t launch_t(ConvParams p, hipStream_t st) {
  constexpr int LH = 64 / LW;
  constexpr int TH = LH * R, TW = LW * CC;
  p.tiles_x = (p.wo + TW - 1) / TW;
  p.tiles_y = (p.ho + TH - 1) / TH;
  p.n_ftiles = (p.n_groups + WF * NG - 1) / (WF * NG);
  const size_t nb = static_cast<size_t>(p.n_ftiles) * p.tiles_x * p.tiles_y * p.n;
  if (nb == 0 || nb > 0x7FFFFFFFull) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((pp_conv3x3_kernel<LIB, S, D, R, CC, LW, NG, WF, WS, CCH, TA>), dim3(static_cast<uint32_t>(nb)),
                     dim3(WF * WS * 64), 0, st, p);
  return hipGetLastError();
}

template <int LIB, int S, int D, class TA>
hipError_t launch_sd(const ConvPlan& plan, ConvParams p, hipStream_t st) {
  constexpr int CCH = (S == 2) ? 4 : 8;   // stride-2 halo tiles are ~4x larger
  switch (plan.recipe) {
    case 0:  // large maps: 16x32 tile, 4 waves along filters
      return launch_t<LIB, S, D, 2, 4, 8, 1, 4, 1, CCH, TA>(p, st);
    case 1:  // medium maps: 16x32 tile, 2 filter waves x 2 channel-split waves
      return launch_t<LIB, S, D, 2, 4, 8, 1, 2, 2, CCH, TA>(p, st);
    case 2:  // small maps: 16x16 tile, 1 filter wave x 4 channel-split waves
      return launch_t<LIB, S, D, 2, 2, 8, 1, 1, 4, CCH, TA>(p, st);
    default:
      return hipErrorInvalidValue;
  }
}

template <int LIB, class TA>
hipError_t launch_lib(const ConvPlan& plan, const ConvParams& p, hipStream_t st) {
  if (p.stride == 1 && p.dil == 1) return launch_sd<LIB, 1, 1, TA>(plan, p, st);
  if (p.stride == 2 && p.dil == 1) return launch_sd<LIB, 2, 1, TA>(plan, p, st);
  if (p.stride == 1 && p.dil == 2) return launch_sd<LIB, 1, 2, TA>(plan, p, st);
  if (p.stride == 2 && p.dil == 2) return launch_sd<LIB, 2, 2, TA>(plan, p, st);
  return hipErrorInvalidValue;
}

}  // namespace

ConvPlan plan_conv(const ConvParams& p, int lib) {
  (void)lib;
  ConvPlan plan;
  const long pix = static_cast<long>(p.ho) * p.wo;
  if (pix >= 100L * 100L)
    plan.recipe = 0;
  else if (pix >= 40L * 40L)
    plan.recipe = 1;
  else
    plan.recipe = 2;
  return plan;
}

hipError_t launch_conv(int lib, const ConvPlan& plan, const ConvParams& p, bool bf16_act, hipStream_t st) {
  if (bf16_act) {
    if (lib == kLibCanon8) return launch_lib<kLibCanon8, uint16_t>(plan, p, st);
    if (lib == kLibDense9) return launch_lib<kLibDense9, uint16_t>(plan, p, st);
    return launch_lib<kLibGeneric, uint16_t>(plan, p, st);
  }
  if (lib == kLibCanon8) return launch_lib<kLibCanon8, float>(plan, p, st);
  if (lib == kLibDense9) return launch_lib<kLibDense9, float>(plan, p, st);
  return launch_lib<kLibGeneric, float>(plan, p, st);
}

}  // namespace pp
