// conv_pp_kernel.hpp -- the pattern/connectivity-pruned 3x3 convolution
// kernel template for gfx950 (included by the per-library .hip files).
//
// One launch computes y = act(conv(x, W_pruned) + b) for a PPK1-packed layer
// (pattern + connectivity pruning, Sec. 2; compact storage and filter
// reorder, Sec. 3; conv fused with bias and activation, Sec. 3).
//
// Mapping to CDNA4:
//   * A workgroup owns one spatial output tile of one image and WF slot
//     groups (8 packed filters each, one group per wave).  Its input halo
//     tile is staged from HBM into LDS one chunk of CCH = WS*CPW input
//     channels at a time (coalesced along rows, zero-filled outside the
//     image) and shared by every filter of the workgroup.
//   * Lanes are output pixels: each lane owns an R x CC block of outputs for
//     the 8 filters of its wave, so the 3x3 neighbourhood it needs for one
//     input channel (the "patch") is read from LDS once and reused by every
//     kept kernel of that channel.
//   * Everything that depends on the sparsity structure is wave-uniform: the
//     per-(group, channel) code word, the weight offset and the weights are
//     scalar loads into SGPRs, and the pattern selects a code path through a
//     uniform branch whose tap offsets are compile-time constants.  No lane
//     ever diverges on the pruning structure.
//   * Software pipelining: code words for the wave's channels of a chunk are
//     fetched before the chunk is staged; the weights and the patch of
//     channel k+1 are in flight while channel k is computed.
//   * WS waves of a workgroup split each chunk's channels; their partial sums
//     are combined through LDS by a fixed binary tree, so results are
//     deterministic.
#pragma once

#ifndef __HIPCC_RTC__   // (the run-time compiler, which provides these itself)
#include <hip/hip_runtime.h>

#include <cstdint>
#endif

#include "conv_pp.hpp"

namespace pp {
namespace kern {

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
__device__ __forceinline__ uint32_t to_bf16_bits(float v) {
  uint32_t u = __float_as_uint(v);
  u += 0x7FFFu + ((u >> 16) & 1u);   // round to nearest even (finite values)
  return u >> 16;
}

// wait until every outstanding LDS and scalar-memory load has returned
__device__ __forceinline__ void wait_lgkm() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// workgroup barrier for LDS hand-off without a memory fence: the caller has
// already waited for the LDS writes that matter (its own ds ops complete in
// order; DMA writes via an explicit vmcnt wait)
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// LDS pointers as 32-bit LDS byte addresses and back
typedef __attribute__((address_space(3))) void* lds_void_ptr;
template <class T>
__device__ __forceinline__ uint32_t lds_addr(T* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) T*)p));
}
__device__ __forceinline__ lds_void_ptr lds_ptr(uint32_t a) { return (lds_void_ptr)(uintptr_t)a; }

// The compile-time 8-entry library of 4-tap patterns behind the "canonical"
// kernels: the canonical library (0x03A, ...), or, in a module compiled at
// run time for a layer's own 4-tap library (PP_JIT_LIBRARY, up to 8 masks,
// padded with the last one), that library.
#ifdef PP_JIT_LIBRARY
constexpr uint32_t kCanon8[8] = {PP_JIT_LIBRARY};
#else
constexpr uint32_t kCanon8[8] = {0x03A, 0x0B2, 0x0B8, 0x09A, 0x01B, 0x036, 0x0D8, 0x1B0};
#endif

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

// the same dispatch on the 3-bit pattern code held at bit SH of a code word,
// as a tree of bit tests on the word itself (no extraction, no compares).
// Each level re-reads the word in place through an empty asm, so its test
// stays a scalar bit test right before its branch (tests hoisted above the
// tree become 64-bit condition masks and extra instructions).
template <int BIT>
__device__ __forceinline__ bool sbit(uint32_t& cw) {
  asm volatile("" : "+s"(cw));
  return (cw >> BIT) & 1u;
}
template <int SH, int S, int D, int R, int CC, int PR, int PC>
__device__ __forceinline__ void apply_canon8_bits(uint32_t cw, float (&acc)[R][CC], const float (&pt)[PR][PC],
                                                  float w0, float w1, float w2, float w3) {
  if (sbit<SH + 2>(cw)) {
    if (sbit<SH + 1>(cw)) {
      if (sbit<SH>(cw))
        apply4<kCanon8[7], S, D>(acc, pt, w0, w1, w2, w3);
      else
        apply4<kCanon8[6], S, D>(acc, pt, w0, w1, w2, w3);
    } else {
      if (sbit<SH>(cw))
        apply4<kCanon8[5], S, D>(acc, pt, w0, w1, w2, w3);
      else
        apply4<kCanon8[4], S, D>(acc, pt, w0, w1, w2, w3);
    }
  } else {
    if (sbit<SH + 1>(cw)) {
      if (sbit<SH>(cw))
        apply4<kCanon8[3], S, D>(acc, pt, w0, w1, w2, w3);
      else
        apply4<kCanon8[2], S, D>(acc, pt, w0, w1, w2, w3);
    } else {
      if (sbit<SH>(cw))
        apply4<kCanon8[1], S, D>(acc, pt, w0, w1, w2, w3);
      else
        apply4<kCanon8[0], S, D>(acc, pt, w0, w1, w2, w3);
    }
  }
}

// generic library: taps tested one by one against the runtime mask
template <int S, int D, int R, int CC, int PR, int PC>
__device__ __forceinline__ void apply_generic(uint32_t mask, float (&acc)[R][CC], const float (&pt)[PR][PC],
                                              const uint8_t* blob, uint32_t off_w, uint32_t k, uint32_t n_wt,
                                              bool bf16w) {
  uint32_t q = 0;
  const uint32_t last = n_wt ? n_wt - 1 : 0u;   // clamp: never read past the weights
#define PP_TAP(T)                                                \
  if (mask & (1u << T)) {                                        \
    const uint32_t kq = min(k + q, last);                        \
    float wv;                                                    \
    if (bf16w) {                                                 \
      uint32_t u = sload<uint32_t>(blob, (off_w + 2 * kq) & ~3u); \
      wv = (kq & 1) ? bf16_hi(u) : bf16_lo(u);                   \
    } else {                                                     \
      wv = sload<float>(blob, off_w + 4 * kq);                   \
    }                                                            \
    fma_tap<T, S, D>(acc, pt, wv);                               \
    ++q;                                                         \
  }
  PP_TAP(0) PP_TAP(1) PP_TAP(2) PP_TAP(3) PP_TAP(4) PP_TAP(5) PP_TAP(6) PP_TAP(7) PP_TAP(8)
#undef PP_TAP
}

// blockIdx -> logical block so that consecutive logical blocks (which share
// the same input tile) land on the same XCD: the dispatcher sends block b to
// XCD b % 8, and each XCD has its own L2.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t b, uint32_t nb) {
  const uint32_t x = b & 7u, local = b >> 3;
  const uint32_t q0 = nb >> 3, r = nb & 7u, q1 = q0 + (r ? 1u : 0u);
  return x < r ? x * q1 + local : r * q1 + (x - r) * q0 + local;
}

// compile-time geometry of one tiling
template <int S, int D, int R, int CC, int LW, int WF, int WS, int CPW, bool DMA, bool LDSW>
struct Geo {
  static constexpr int LH = 64 / LW;
  static constexpr int TH = LH * R, TW = LW * CC;          // output tile
  static constexpr int PR = (R - 1) * S + 2 * D + 1;       // patch rows
  static constexpr int PC = (CC - 1) * S + 2 * D + 1;      // patch cols
  static constexpr int TIH = (TH - 1) * S + 2 * D + 1;     // input tile rows
  static constexpr int TIW = (TW - 1) * S + 2 * D + 1;     // input tile cols
  static constexpr int LSTR = (TIW + 3) / 4 * 4;           // LDS row stride (floats)
  static constexpr int NW = WF * WS;                       // waves per workgroup
  static constexpr int CCH = WS * CPW;                     // channels per chunk
  // DMA staging writes whole 64-float segments; a channel's region is padded
  // so that its NQ segments split evenly over the NW waves
  static constexpr int SEG = 64 * NW;
  static constexpr int CHSTR = DMA ? (TIH * LSTR + SEG - 1) / SEG * SEG : TIH * LSTR;
  static constexpr int NQ = CHSTR / 64;                    // DMA segments per channel
  static constexpr int NQW = NQ / NW;                      // ... per wave
  static constexpr int LOADS = CCH * NQW;                  // DMA loads per wave per chunk
  static constexpr int NACC = 8 * R * CC;
  // canonical library, fp32: next to each staged input chunk, the chunk's
  // weights of every slot group expanded to a fixed [channel][slot][4] layout
  // (pruned slots zero); the metadata (CCH woff entries, then 2*CCH code
  // dwords from index 32) sits in a ring of 4 buffers of 64 dwords per group
  static constexpr int WEXP = CCH * 32;                    // expanded weights per group
  static constexpr int GDATA = LDSW ? WF * WEXP : 0;
  static constexpr int META = LDSW ? 4 * WF * 64 : 0;
  static constexpr int BUF = CCH * CHSTR + GDATA;          // one staged chunk
  static constexpr int RED = (WS > 1) ? (WS / 2) * WF * NACC * 64 : 0;
  // lds0 = max(chunk, partial-sum exchange); DMA adds a second chunk buffer
  static constexpr int LDS_FLOATS = (BUF > RED ? BUF : RED) + (DMA ? BUF : 0) + META;
  static constexpr int VW = ((CC * S) % 4 == 0) ? 4 : (((CC * S) % 2 == 0) ? 2 : 1);
  static constexpr int N4 = (VW == 4) ? PC / 4 : 0;
  static constexpr int N2 = (VW >= 2) ? (PC - 4 * N4) / 2 : 0;
  static constexpr int N1 = PC - 4 * N4 - 2 * N2;
  static constexpr bool fits = LDS_FLOATS * 4 <= 160 * 1024 && LW * LH == 64 && (WS & (WS - 1)) == 0 &&
                               CCH <= 16 && CCH % 2 == 0;
};

template <int LIB, int S, int D, int R, int CC, int LW, int WF, int WS, int CPW, class TA>
__global__ __launch_bounds__(WF* WS * 64) void pp_conv3x3_kernel(ConvParams a) {
  constexpr bool WBF = sizeof(TA) == 2;   // bf16 weights with bf16 activations
  constexpr bool DMA = !WBF;              // fp32: stage with direct buffer->LDS loads
  constexpr bool LDSW = DMA && LIB == kLibCanon8;   // code words + weights staged in LDS too
  using G = Geo<S, D, R, CC, LW, WF, WS, CPW, DMA, LDSW>;
  constexpr int PR = G::PR, PC = G::PC, TIH = G::TIH, TIW = G::TIW, LSTR = G::LSTR, CHSTR = G::CHSTR;
  constexpr int CCH = G::CCH, NACC = G::NACC, NW = G::NW;
  static_assert(G::fits, "tiling does not fit");

  // DMA path: two distinct LDS arrays (static buffer selection lets the
  // compiler see that loads into one never alias reads of the other);
  // lds0 also holds the single buffer of the register path and the
  // partial-sum exchange of the split-channel waves.
  constexpr int LDS0 = G::BUF > G::RED ? G::BUF : G::RED;
  __shared__ __attribute__((aligned(16))) float lds0[LDS0];
  __shared__ __attribute__((aligned(16))) float lds1[DMA ? G::BUF : 1];
  __shared__ __attribute__((aligned(16))) uint32_t ldsm[LDSW ? G::META : 1];
  float* const lds = lds0;

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

  const int oy0 = ty * G::TH, ox0 = tx * G::TW;
  const int iy0 = oy0 * S - a.pad, ix0 = ox0 * S - a.pad;
  const int grp = ft * WF + wf;               // this wave's slot group
  const bool has_grp = grp < a.n_groups;      // wave-uniform

  const TA* __restrict__ x = static_cast<const TA*>(a.x) + static_cast<size_t>(img) * a.c_in * a.h * a.w;
  const uint8_t* blob = a.blob;
  // this image of x as a buffer resource: loads past its end return 0
  const uint32_t img_bytes = static_cast<uint32_t>(a.c_in) * a.h * a.w * sizeof(TA);
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<TA*>(x), static_cast<short>(0), static_cast<int>(img_bytes), 0x00020000);
  const uint32_t chan_bytes = static_cast<uint32_t>(a.h) * a.w * sizeof(TA);
  const int n_chunks = (a.c_in + CCH - 1) / CCH;
  // the blob as a buffer resource (group-data staging): reads past its end return 0
  const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(blob), static_cast<short>(0), static_cast<int>(a.blob_bytes), 0x00020000);
  const int sgrp = has_grp ? grp : 0;   // clamped group for address arithmetic

  float acc[8][R][CC];
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int q = 0; q < CC; ++q) acc[s][r][q] = 0.0f;

  const int lane_off = (ly * R * S) * LSTR + lx * CC * S;

  // ---- staging (fp32): every wave issues segments m = wid + NW*t of every
  // channel of a chunk; lane l of segment m stages element q = 64m + l of the
  // channel's LDS region (row q / LSTR, col q % LSTR).  Its byte offset in
  // the channel is fixed for the whole kernel; padding and out-of-image
  // elements get an offset past the buffer, which the hardware returns as 0.
  uint32_t qoff[DMA ? G::NQW : 1];
  if constexpr (DMA) {
#pragma unroll
    for (int t = 0; t < G::NQW; ++t) {
      const int q = 64 * (wid + NW * t) + lane;
      const int row = q / LSTR, col = q % LSTR;
      const int gy = iy0 + row, gx = ix0 + col;
      const bool ok = row < TIH && col < TIW && gy >= 0 && gy < a.h && gx >= 0 && gx < a.w;
      qoff[t] = ok ? (static_cast<uint32_t>(gy) * a.w + gx) * 4u : 0x80000000u;
    }
  }
  auto stage_dma = [&](int chunk, float* base) __attribute__((always_inline)) {
    // launder the LDS base (as a 32-bit LDS address): otherwise the compiler
    // hoists all CCH*NQW destination addresses out of the chunk loop and
    // spills SGPRs
    uint32_t lb = lds_addr(base);
    asm volatile("" : "+s"(lb));
#pragma unroll
    for (int ch = 0; ch < CCH; ++ch) {
      // channels past c_in read at offset >= the buffer size: zeros
      const uint32_t cofs = static_cast<uint32_t>(min(chunk * CCH + ch, a.c_in)) * chan_bytes;
#pragma unroll
      for (int t = 0; t < G::NQW; ++t)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, lds_ptr(lb + 4u * (ch * CHSTR + 64 * (wid + NW * t))), 4,
                                                 qoff[t], cofs, 0, 0);
    }
  };

  // ---- group data (canonical library, fp32), staged by wave (wf, 0) for its
  // slot group.  Metadata of a chunk: woff entries in lanes 0..CCH-1, code
  // dwords in lanes 32..32+2*CCH-1 of one 64-dword DMA.
  auto stage_meta = [&](int chunk) __attribute__((always_inline)) {
    uint32_t mb = lds_addr(ldsm + ((chunk & 3) * WF + wf) * 64);
    asm volatile("" : "+s"(mb));
    const uint32_t e0 = static_cast<uint32_t>(sgrp) * a.c_in + chunk * CCH;
    uint32_t off;
    if (lane < CCH)
      off = a.off_woff + 4u * (e0 + lane);
    else if (lane >= 32 && lane < 32 + 2 * CCH)
      off = a.off_codes + 8u * (e0 + ((lane - 32) >> 1)) + 4u * ((lane - 32) & 1);
    else
      off = 0x80000000u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(br, lds_ptr(mb), 4, off, 0, 0, 0);
  };
  // Expanded weights of a chunk (its metadata must already be in LDS): DMA
  // i covers channels 2i, 2i+1; lane l -> channel 2i + l/32, slot (l/4)%8,
  // tap l%4.  A kept slot's weights sit at rank popcount(kept & (2^s-1)) of
  // its channel's entry; pruned slots and channels past c_in load zero.
  auto stage_wexp = [&](int chunk, float* base) __attribute__((always_inline)) {
    const uint32_t* meta = ldsm + ((chunk & 3) * WF + wf) * 64;
    uint32_t wb = lds_addr(base + CCH * CHSTR + wf * G::WEXP);
    asm volatile("" : "+s"(wb));
    const int s = (lane >> 2) & 7, q = lane & 3;
    uint32_t wo[CCH / 2];
#pragma unroll
    for (int i = 0; i < CCH / 2; ++i) wo[i] = meta[2 * i + (lane >> 5)];
#pragma unroll
    for (int i = 0; i < CCH / 2; ++i) {
      const int c = chunk * CCH + 2 * i + (lane >> 5);
      const uint32_t kmask = wo[i] >> 24;
      const uint32_t rank = __builtin_popcount(kmask & ((1u << s) - 1u));
      const bool ok = c < a.c_in && ((kmask >> s) & 1u);
      const uint32_t off = ok ? a.off_w + 4u * ((wo[i] & 0xFFFFFFu) + 4u * rank + q) : 0x80000000u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(br, lds_ptr(wb + 4u * 64 * i), 4, off, 0, 0, 0);
    }
  };

  // ---- staging (bf16): wave w stages rows [w*RPW, (w+1)*RPW) of the chunk's
  // CCH x TIH rows (wave-uniform row coordinates), lanes cover the columns and
  // convert to fp32; all loads of a lane are issued before its LDS writes.
  constexpr int NCB = (TIW + 63) / 64;
  constexpr int RPW = (CCH * TIH + NW - 1) / NW;
  auto stage_regs = [&](int cb) __attribute__((always_inline)) {
    // opaque copy of the chunk index: keeps the compiler from hoisting the
    // per-row arithmetic out of the chunk loop (it would pin ~2 SGPRs per
    // staged row for the whole kernel)
    int cbo = cb;
    asm volatile("" : "+s"(cbo));
    float v[RPW][NCB];
#pragma unroll
    for (int k = 0; k < RPW; ++k) {
      const int row = wid * RPW + k + (cbo - cb);
      const int ch = row / TIH, i = row % TIH;
      const int c = cb + ch, gy = iy0 + i;
      const bool row_ok = row < CCH * TIH && c < a.c_in && gy >= 0 && gy < a.h;   // wave-uniform
      const uint32_t rbase = (static_cast<uint32_t>(c) * a.h + gy) * static_cast<uint32_t>(a.w);
#pragma unroll
      for (int m = 0; m < NCB; ++m) {
        const int gx = ix0 + lane + 64 * m;
        const bool ok = row_ok && lane + 64 * m < TIW && gx >= 0 && gx < a.w;
        const uint32_t off = ok ? (rbase + gx) * sizeof(TA) : 0x80000000u;
        if (sizeof(TA) == 2)
          v[k][m] = __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(xr, off, 0, 0)) << 16);
        else
          v[k][m] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xr, off, 0, 0));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    float* dst = lds + wid * RPW * LSTR + lane;
#pragma unroll
    for (int k = 0; k < RPW; ++k) {
      if (wid * RPW + k + (cbo - cb) < CCH * TIH) {
#pragma unroll
        for (int m = 0; m < NCB; ++m)
          if (lane + 64 * m < TIW) dst[k * LSTR + 64 * m] = v[k][m];
      }
    }
  };

  // ---- one chunk: every kept kernel of this wave's 8 filters on the wave's
  // CPW channels of the chunk held in LDS buffer `buf`
  auto load_patch = [&](float(&p)[PR][PC], const float* src) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < PR; ++r) {
      const float* row = src + r * LSTR;
#pragma unroll
      for (int i = 0; i < G::N4; ++i) {
        const float4 v = *reinterpret_cast<const float4*>(row + 4 * i);
        p[r][4 * i] = v.x; p[r][4 * i + 1] = v.y; p[r][4 * i + 2] = v.z; p[r][4 * i + 3] = v.w;
      }
#pragma unroll
      for (int i = 0; i < G::N2; ++i) {
        const float2 v = *reinterpret_cast<const float2*>(row + 4 * G::N4 + 2 * i);
        p[r][4 * G::N4 + 2 * i] = v.x; p[r][4 * G::N4 + 2 * i + 1] = v.y;
      }
#pragma unroll
      for (int i = 0; i < G::N1; ++i) p[r][4 * G::N4 + 2 * G::N2 + i] = row[4 * G::N4 + 2 * G::N2 + i];
    }
  };

  // ---- one chunk, canonical library, fp32: everything the channel loop reads
  // is in LDS -- input patch, metadata, and the weights at fixed
  // [channel][slot] positions, read only for kept slots
  auto compute_chunk_ldsw = [&](int j, const float* base) __attribute__((always_inline)) {
    const int cb = j * CCH;
    const int cl0 = wk * CPW;
    const int nch = has_grp ? max(0, min(CPW, a.c_in - (cb + cl0))) : 0;   // wave-uniform
    if (nch == 0) return;
    const uint32_t* meta = ldsm + ((j & 3) * WF + wf) * 64;
    const float* wexp = base + CCH * CHSTR + wf * G::WEXP;
    uint32_t m_wo = meta[cl0], m_c0 = meta[32 + 2 * cl0], m_c1 = meta[33 + 2 * cl0];
#pragma unroll 1
    for (int k = 0; k < nch; ++k) {
      const uint32_t wo = __builtin_amdgcn_readfirstlane(m_wo);
      const uint32_t cx = __builtin_amdgcn_readfirstlane(m_c0), cy = __builtin_amdgcn_readfirstlane(m_c1);
      if (k + 1 < nch) {
        m_wo = meta[cl0 + k + 1];
        m_c0 = meta[32 + 2 * (cl0 + k + 1)];
        m_c1 = meta[33 + 2 * (cl0 + k + 1)];
      }
      const uint32_t kept = wo >> 24;   // bit s: slot s has a kept kernel
      if (kept == 0) continue;
      float p[PR][PC];
      load_patch(p, base + (cl0 + k) * CHSTR + lane_off);
      const float4* wc = reinterpret_cast<const float4*>(wexp + (cl0 + k) * 32);
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        if (!((kept >> s) & 1u)) continue;
        const float4 w = wc[s];
        const uint32_t pid = ((s < 4 ? cx : cy) >> (8 * (s & 3))) & 0xFFu;
        apply_canon8<S, D>(pid, acc[s], p, w.x, w.y, w.z, w.w);
      }
    }
  };

  auto compute_chunk = [&](int cb, const float* base) __attribute__((always_inline)) {
    const int cl0 = wk * CPW;
    const int nch = has_grp ? max(0, min(CPW, a.c_in - (cb + cl0))) : 0;   // wave-uniform
    // code word and woff of the first channel; the loop prefetches the next
    uint32_t e = static_cast<uint32_t>(has_grp ? grp : 0) * a.c_in + min(cb + cl0, a.c_in - 1);
    uint2 cw_next = sload<uint2>(blob, a.off_codes + 8 * e);
    uint32_t wo_next = sload<uint32_t>(blob, a.off_woff + 4 * e);
#pragma unroll 1
    for (int k = 0; k < nch; ++k) {
      const uint2 cw = cw_next;
      const uint32_t wo = wo_next;
      if (k + 1 < nch) {
        ++e;
        cw_next = sload<uint2>(blob, a.off_codes + 8 * e);
        wo_next = sload<uint32_t>(blob, a.off_woff + 4 * e);
      }
      const uint32_t kept = wo >> 24;   // bit s: slot s has a kept kernel
      if (kept == 0) continue;
      // first weight of the entry.  Canonical library: clamped so that the
      // unconditional 4-weight read of every slot stays inside the weight
      // array (plus the >= 32 bytes that follow it); other libraries read
      // kernel by kernel with clamped reads, and their kernels may hold fewer
      // than 4 weights, so the entry's own offset is used (a clamp assuming
      // 4 per kernel would move it)
      const uint32_t nk4 = static_cast<uint32_t>(__builtin_popcount(kept)) * 4u;
      const uint32_t w0 = LIB == kLibCanon8 ? min(wo & 0xFFFFFFu, a.n_wt - min(a.n_wt, nk4))
                                            : min(wo & 0xFFFFFFu, a.n_wt);
      // patch: the lane's input neighbourhood for this channel
      float p[PR][PC];
      load_patch(p, base + (cl0 + k) * CHSTR + lane_off);
      if (LIB == kLibCanon8) {
        // weights of all 8 slots, issued together: slot s reads the kernel at
        // rank popcount(kept & (2^s - 1)) of the entry (4 weights each)
        float4 wv[8];
        const uint32_t wbyte = a.off_w + (WBF ? 2u : 4u) * w0;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const uint32_t rank = static_cast<uint32_t>(__builtin_popcount(kept & ((1u << s) - 1u)));
          if (WBF) {
            const uint2 u = sload<uint2>(blob, wbyte + 8u * rank);
            wv[s] = make_float4(bf16_lo(u.x), bf16_hi(u.x), bf16_lo(u.y), bf16_hi(u.y));
          } else {
            wv[s] = sload<float4>(blob, wbyte + 16u * rank);
          }
        }
        // materialise all weights here: one wait for the whole group-channel
        // instead of a load + wait sunk into every dispatch branch
#pragma unroll
        for (int s = 0; s < 8; ++s) asm volatile("" ::"s"(wv[s].x), "s"(wv[s].y), "s"(wv[s].z), "s"(wv[s].w));
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          if (!((kept >> s) & 1u)) continue;
          const uint32_t pid = ((s < 4 ? cw.x : cw.y) >> (8 * (s & 3))) & 0xFFu;
          apply_canon8<S, D>(pid, acc[s], p, wv[s].x, wv[s].y, wv[s].z, wv[s].w);
        }
      } else {
        uint32_t kk = w0;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          if (!((kept >> s) & 1u)) continue;
          const uint32_t pid = ((s < 4 ? cw.x : cw.y) >> (8 * (s & 3))) & 0xFFu;
          if (LIB == kLibDense9) {
            float w9[9];
            if (WBF) {
              const uint32_t kc = min(kk, a.n_wt >= 10 ? a.n_wt - 10 : 0u);
              const uint4 u = sload<uint4>(blob, a.off_w + 2 * kc);
              const uint32_t u4 = sload<uint32_t>(blob, a.off_w + 2 * kc + 16);
              w9[0] = bf16_lo(u.x); w9[1] = bf16_hi(u.x); w9[2] = bf16_lo(u.y); w9[3] = bf16_hi(u.y);
              w9[4] = bf16_lo(u.z); w9[5] = bf16_hi(u.z); w9[6] = bf16_lo(u.w); w9[7] = bf16_hi(u.w);
              w9[8] = bf16_lo(u4);
              kk += 10;
            } else {
              const uint32_t kc = min(kk, a.n_wt >= 9 ? a.n_wt - 9 : 0u);
              const float4 u = sload<float4>(blob, a.off_w + 4 * kc);
              const float4 v = sload<float4>(blob, a.off_w + 4 * kc + 16);
              const float z = sload<float>(blob, a.off_w + 4 * kc + 32);
              w9[0] = u.x; w9[1] = u.y; w9[2] = u.z; w9[3] = u.w;
              w9[4] = v.x; w9[5] = v.y; w9[6] = v.z; w9[7] = v.w; w9[8] = z;
              kk += 9;
            }
            fma_tap<0, S, D>(acc[s], p, w9[0]);
            fma_tap<1, S, D>(acc[s], p, w9[1]);
            fma_tap<2, S, D>(acc[s], p, w9[2]);
            fma_tap<3, S, D>(acc[s], p, w9[3]);
            fma_tap<4, S, D>(acc[s], p, w9[4]);
            fma_tap<5, S, D>(acc[s], p, w9[5]);
            fma_tap<6, S, D>(acc[s], p, w9[6]);
            fma_tap<7, S, D>(acc[s], p, w9[7]);
            fma_tap<8, S, D>(acc[s], p, w9[8]);
          } else {
            const uint32_t pc = min(pid, static_cast<uint32_t>(a.n_patterns - 1));
            const uint32_t mw = sload<uint32_t>(blob, (a.off_masks + 2 * pc) & ~3u);
            const uint32_t mask = ((pc & 1u) ? (mw >> 16) : mw) & 0x1FFu;
            apply_generic<S, D>(mask, acc[s], p, blob, a.off_w, kk, a.n_wt, WBF);
            const uint32_t nt = __builtin_popcount(mask);
            kk += WBF ? ((nt + 1u) & ~1u) : nt;
          }
        }
      }
    }
  };

  if constexpr (DMA) {
    // double-buffered: chunk j+1 streams into one LDS array while chunk j is
    // computed from the other (two chunks per trip keep the selection
    // static).  Step j: wait for everything issued so far (chunk j's input
    // and group data), one barrier (chunk j visible; chunk j-1 no longer
    // read), issue chunk j+1 (and the metadata of chunk j+3), compute j.
    const bool gstager = LDSW && wk == 0;   // this wave stages its group's data
    if (gstager) {
      stage_meta(0);
      if (1 < n_chunks) stage_meta(1);
      if (2 < n_chunks) stage_meta(2);
      __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): metadata of chunks 0..2
    }
    stage_dma(0, lds0);
    if (gstager) stage_wexp(0, lds0);
    auto step = [&](int j, const float* cur, float* nxt) __attribute__((always_inline)) {
      __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
      // plain s_barrier: __syncthreads() would make the compiler wait for
      // memory operations that are intentionally still in flight
      lds_barrier();
      if (j + 1 < n_chunks) {
        stage_dma(j + 1, nxt);
        if (gstager) {
          stage_wexp(j + 1, nxt);
          if (j + 3 < n_chunks) stage_meta(j + 3);
        }
      }
      if constexpr (LDSW)
        compute_chunk_ldsw(j, cur);
      else
        compute_chunk(j * CCH, cur);
    };
    for (int j = 0; j < n_chunks; j += 2) {
      step(j, lds0, lds1);
      if (j + 1 < n_chunks) step(j + 1, lds1, lds0);
    }
  } else {
    for (int cb = 0; cb < a.c_in; cb += CCH) {
      __syncthreads();   // the previous chunk's LDS reads are done
      stage_regs(cb);
      __syncthreads();
      compute_chunk(cb, lds0);
    }
  }

  // ---- combine the WS channel-split partial sums: fixed binary tree
  if (WS > 1) {
#pragma unroll
    for (int half = WS / 2; half >= 1; half /= 2) {
      __syncthreads();
      if (wk >= half && wk < 2 * half) {
        float* dst = lds + static_cast<size_t>((wk - half) * WF + wf) * NACC * 64 + lane;
        int i = 0;
#pragma unroll
        for (int s = 0; s < 8; ++s)
#pragma unroll
          for (int r = 0; r < R; ++r)
#pragma unroll
            for (int q = 0; q < CC; ++q, ++i) dst[i * 64] = acc[s][r][q];
      }
      __syncthreads();
      if (wk < half) {
        const float* src = lds + static_cast<size_t>(wk * WF + wf) * NACC * 64 + lane;
        int i = 0;
#pragma unroll
        for (int s = 0; s < 8; ++s)
#pragma unroll
          for (int r = 0; r < R; ++r)
#pragma unroll
            for (int q = 0; q < CC; ++q, ++i) acc[s][r][q] += src[i * 64];
      }
    }
    if (wk > 0) return;
  }
  if (!has_grp) return;

  // ---- epilogue: + bias, activation, store to the original channel order
  TA* __restrict__ y = static_cast<TA*>(a.y) + static_cast<size_t>(img) * a.c_out * a.ho * a.wo;
  const bool relu = (a.flags & PP_RELU) != 0;
  const int oxl = ox0 + lx * CC;
  const bool vec = (CC % 4 == 0) && (a.wo % 4 == 0) &&
                   (reinterpret_cast<uintptr_t>(a.y) % (4 * sizeof(TA)) == 0);   // aligned vector stores
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
      TA* row = y + (static_cast<size_t>(o) * a.ho + oy) * a.wo;
      float v[CC];
#pragma unroll
      for (int q = 0; q < CC; ++q) {
        v[q] = acc[s][r][q] + bias;
        if (relu) v[q] = fmaxf(v[q], 0.0f);
      }
      if (vec && oxl + CC <= a.wo) {
#pragma unroll
        for (int q = 0; q < CC; q += 4) {
          if (WBF) {
            uint2 u;
            u.x = to_bf16_bits(v[q]) | (to_bf16_bits(v[q + 1]) << 16);
            u.y = to_bf16_bits(v[q + 2]) | (to_bf16_bits(v[q + 3]) << 16);
            *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(row) + oxl + q) = u;
          } else {
            *reinterpret_cast<float4*>(reinterpret_cast<float*>(row) + oxl + q) =
                make_float4(v[q], v[q + 1], v[q + 2], v[q + 3]);
          }
        }
      } else {
#pragma unroll
        for (int q = 0; q < CC; ++q) {
          if (oxl + q < a.wo) {
            if (WBF)
              reinterpret_cast<uint16_t*>(row)[oxl + q] = static_cast<uint16_t>(to_bf16_bits(v[q]));
            else
              reinterpret_cast<float*>(row)[oxl + q] = v[q];
          }
        }
      }
    }
  }
}

#ifndef __HIPCC_RTC__   // host side
// ---------------------------------------------------------------------------
// host side: one tiling = one Recipe; launch helpers
// ---------------------------------------------------------------------------
template <int LIB, int S, int D, int R, int CC, int LW, int WF, int WS, int CPW, class TA>
hipError_t launch_tiling(ConvParams p, hipStream_t st) {
  using G = Geo<S, D, R, CC, LW, WF, WS, CPW, sizeof(TA) == 4, sizeof(TA) == 4 && LIB == kLibCanon8>;
  if constexpr (!G::fits) {
    return hipErrorInvalidConfiguration;
  } else {
    p.tiles_x = (p.wo + G::TW - 1) / G::TW;
    p.tiles_y = (p.ho + G::TH - 1) / G::TH;
    p.n_ftiles = (p.n_groups + WF - 1) / WF;
    const size_t nb = static_cast<size_t>(p.n_ftiles) * p.tiles_x * p.tiles_y * p.n;
    if (nb == 0 || nb > 0x7FFFFFFFull) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((pp_conv3x3_kernel<LIB, S, D, R, CC, LW, WF, WS, CPW, TA>), dim3(static_cast<uint32_t>(nb)),
                       dim3(WF * WS * 64), 0, st, p);
    return hipGetLastError();
  }
}

#endif

}  // namespace kern
}  // namespace pp
