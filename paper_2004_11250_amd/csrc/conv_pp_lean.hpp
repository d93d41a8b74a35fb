// conv_pp_lean.hpp -- pattern/connectivity-pruned 3x3 convolution for the
// canonical 8-pattern library, fp32, "lean" form (gfx950).
//
// Same result as the wave-pipeline kernel (pattern + connectivity pruning,
// Sec. 2; compact storage and filter reorder, Sec. 3; conv fused with bias
// and activation, Sec. 3) and the same per-wave organisation: a workgroup
// owns one output tile of one image and one slot group of 8 reordered
// filters; its WS waves walk contiguous ranges of the input channels, each
// with a private LDS ring of NS channels that LDS-DMA loads fill; lanes
// are output pixels (R x CC per lane), so a kernel's pattern is wave-uniform
// and selects a code path with compile-time tap offsets.
//
// What differs is everything around the channel loop, which on MI355X cost
// more than the loop itself for the layer sizes of the evaluated networks
// (a few thousand FMAs per wave):
//   * the staging geometry is a compile-time constant (16-byte row DMAs,
//     image width a multiple of 4), so per-lane staging offsets are one
//     constant division each and no branches;
//   * the block decode uses host-computed division magics, not the
//     compiler's run-time division sequences;
//   * the first channel's halo DMAs are issued before the layer metadata is
//     even requested; the metadata of the first channels comes in one scalar
//     load;
//   * the epilogue sums the WS partial blocks with one LDS exchange per pass
//     of slots (two barriers) and stores 16-byte rows.
//
// bf16 activations (BF): the DMAs stage raw bf16 rows (half the bytes), a
// lane reads its patch rows as aligned 4- and 8-byte pieces and widens them
// to fp32 in registers; the weights (bf16 in the blob) are staged as pairs
// and widened per kept slot; accumulation is fp32 and the store rounds once
// to bf16 (round to nearest even).
#pragma once

#include "conv_pp_wave.hpp"

namespace pp {

// q = n / d for n < 2^31 with a host-computed magic (m, l):
// q = (mulhi(n, m) + n) >> l
struct FastDiv {
  uint32_t d = 1, m = 0, l = 0;
};

#ifndef __HIPCC_RTC__
inline FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  f.d = d;
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  f.l = l;
  f.m = static_cast<uint32_t>(((1ull << 32) * ((1ull << l) - d)) / d + 1);
  return f;
}
#endif

struct LeanParams {
  const uint8_t* blob = nullptr;
  const void* x = nullptr;   // float or bf16 (uint16_t) activations
  void* y = nullptr;
  float* part = nullptr;         // channel split over workgroups: partial-sum blocks
  uint32_t h = 0, w = 0, ho = 0, wo = 0;
  uint32_t c_in = 0, c_out = 0;
  uint32_t off_codes = 0, off_woff = 0, off_w = 0, off_bias = 0, off_perm = 0, blob_bytes = 0;
  uint32_t flags = 0;
  uint32_t ksplit = 1;
  const uint8_t* wprep = nullptr;   // prepared weights (PW): [groups][c_in][32] fp32
  FastDiv groups, tiles_x, tiles_y, splits;   // block decode
};

namespace kern {

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv& f) {
  return (__umulhi(n, f.m) + n) >> f.l;
}

// V4: the halo tile is staged by 16-byte DMAs (image width a multiple of
// 4 fp32 / 8 bf16 elements), else by 4-byte DMAs (any width for fp32, even
// for bf16).  Sizes below are in elements unless named otherwise.
// D: the dilation (= the padding): 1, or 2 for fp32; S: the stride: 1, or 2
// for fp32 at dilation 1.
template <int R, int CC, int LW, int WS, bool V4, bool BF = false, int D = 1, int S = 1>
struct LGeo {
  static_assert(D == 1 || (D == 2 && !BF), "dilation 2: fp32 only");
  static_assert(S == 1 || (S == 2 && !BF && D == 1), "stride 2: fp32 at dilation 1 only");
  static constexpr int ES = BF ? 2 : 4;                 // element bytes
  static constexpr int LH = 64 / LW;
  static constexpr int TH = LH * R, TW = LW * CC;       // output tile
  static constexpr int PR = (R - 1) * S + 2 * D + 1, PC = (CC - 1) * S + 2 * D + 1;   // patch of a lane
  static constexpr int TIH = (TH - 1) * S + 2 * D + 1;  // staged rows
  // the staged columns start SH columns before the tile's first input
  // column: fp32 16-byte staging at a multiple of 4 (SH 4 - D), fp32 4-byte
  // staging at that column (SH 0); bf16 at a multiple of 8 (SH 7) or of 2
  // (SH 3), so that a lane's first input element sits one after a dword
  // boundary and its row reads are aligned pieces
  static constexpr int SH = V4 ? (BF ? 7 : 4 - D) : (BF ? 3 : 0);
  static constexpr int SALIGN = BF ? 8 : 4;
  static constexpr int SWID = ((TW - 1) * S + 2 * D + 1 + SH + SALIGN - 1) / SALIGN * SALIGN;
  // fp32: a lane's patch rows are read with aligned loads of up to VWL
  // floats (the alignment its row start allows)
  static constexpr int VWL = (CC * S) % 4 == 0 ? 4 : ((CC * S) % 2 == 0 ? 2 : 1);
  static constexpr int LSTR = BF ? SWID : wave_row_stride(SWID, R * S);
  static constexpr int AREA = TIH * LSTR;
  static constexpr int DPB = V4 ? 1024 : 256;            // LDS bytes of one DMA instruction
  static constexpr int EPD = DPB / ES;                   // elements per DMA instruction
  static constexpr int NQ = (AREA + EPD - 1) / EPD;      // DMAs per lane and channel
  static constexpr int PATCH = NQ * DPB / 4;             // 4-byte words of a staged channel
  static constexpr int SLOT = PATCH + 64;                // + 8 slots x 4 expanded weights (padded)
  // ring of NS channels (a channel's DMA is issued NS - 1 channels ahead);
  // the smaller rings when four slots would leave a CU fewer than two
  // workgroups of 8 waves, and two slots when three would not fit one
  // workgroup's LDS
  static constexpr int NS = (WS * 4 * SLOT * 4 <= 80 * 1024) ? 4 : (WS * 3 * SLOT * 4 <= 160 * 1024) ? 3 : 2;
  static constexpr int RING = NS * SLOT;
  static constexpr int NACC = 8 * R * CC;
  // partial-sum exchange: SPP slots per pass, as many as fit the LDS that
  // the rings occupy (at least one)
  static constexpr int XPS = R * CC * 64;                // floats of one slot of one wave
  static constexpr int SPP0 = (WS * RING) / (WS * XPS);
  static constexpr int SPP = WS == 1 ? 8 : (SPP0 >= 8 ? 8 : (SPP0 >= 4 ? 4 : (SPP0 >= 2 ? 2 : 1)));
  static constexpr int XCH = WS == 1 ? 0 : WS * SPP * XPS;
  static constexpr int LDS_FLOATS = WS * RING > XCH ? WS * RING : XCH;
  static constexpr bool fits = LDS_FLOATS * 4 <= 160 * 1024 && WS >= 1 && WS <= 16 && LW * LH == 64 && TW % 4 == 0 &&
                               (!BF || (CC % 2 == 0 && (!V4 || TW % 8 == 0)));
};

// bf16 bits to fp32
__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }
__device__ __forceinline__ uint32_t bf_rne(float f) {   // fp32 to bf16 bits, round to nearest even (finite)
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// one bf16 patch row of a lane: elements [0, PC) of the lane's row, which
// starts at element index st of the staged row (st odd: it sits one after a
// dword boundary) at LDS byte address rb + 2 st.  Read as the dword holding
// (st - 1, st), then 8-byte pieces while they fit (st + 1 is a multiple of 4
// when CC is a multiple of 4), then dwords.
template <int PC, bool Q8>
__device__ __forceinline__ void read_row_bf(float (&d)[PC], const uint8_t* rb) {
  const uint32_t* w = reinterpret_cast<const uint32_t*>(__builtin_assume_aligned(rb, 4));
  const uint32_t u0 = w[0];
  d[0] = bf_hi(u0);
  int j = 1;
  if constexpr (Q8) {
#pragma unroll
    for (; j + 3 < PC; j += 4) {
      const uint2 u = *reinterpret_cast<const uint2*>(__builtin_assume_aligned(rb + 2 * j + 2, 8));
      d[j] = bf_lo(u.x); d[j + 1] = bf_hi(u.x); d[j + 2] = bf_lo(u.y); d[j + 3] = bf_hi(u.y);
    }
  }
#pragma unroll
  for (; j < PC; j += 2) {
    const uint32_t u = w[(j + 1) / 2];
    d[j] = bf_lo(u);
    if (j + 1 < PC) d[j + 1] = bf_hi(u);
  }
}

// PW: the weights come from a prepared expanded fp32 copy (for bf16 layers
// the bf16 weights widened, exact) by scalar loads into SGPRs (one channel's
// 32 at the end of the step before it), each kept slot's 4 copied to VGPRs
// for its FMAs: no weight DMA and no LDS reads of weights, which relieves the
// LDS path the patch DMAs and reads share
template <int R, int CC, int LW, int WS, bool V4, bool BF = false, bool PW = false, int D = 1, int S = 1>
__global__ __launch_bounds__(WS * 64) void pp_conv3x3_lean_kernel(LeanParams a) {
  using G = LGeo<R, CC, LW, WS, V4, BF, D, S>;
  constexpr uint32_t ES = G::ES;
  constexpr int PR = G::PR, PC = G::PC, LSTR = G::LSTR, NQ = G::NQ, SLOT = G::SLOT, NS = G::NS;
  static_assert(G::fits, "tiling does not fit");
  __shared__ __attribute__((aligned(16))) float lds[G::LDS_FLOATS];

  const int lane = threadIdx.x & 63;
  const int wk = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lx = lane % LW, ly = lane / LW;

  // ---- block -> (image, tile, split, slot group)
  uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
  uint32_t q = fdiv(blk, a.groups);
  const uint32_t grp = blk - q * a.groups.d;
  blk = q;
  q = fdiv(blk, a.splits);
  const uint32_t ks = blk - q * a.splits.d;
  blk = q;
  q = fdiv(blk, a.tiles_x);
  const uint32_t tx = blk - q * a.tiles_x.d;
  blk = q;
  q = fdiv(blk, a.tiles_y);
  const uint32_t ty = blk - q * a.tiles_y.d;
  const uint32_t img = q;

  const int oy0 = ty * G::TH, ox0 = tx * G::TW;
  const int iy0 = oy0 * S - D, ixa = ox0 * S - D - G::SH;   // staged origin

  // ---- this wave's channels: split ks of ksplit, then the wave's part
  const uint32_t kc0 = fdiv(ks * a.c_in, a.splits), kc1 = fdiv((ks + 1) * a.c_in, a.splits);
  const uint32_t per = (kc1 - kc0 + WS - 1) / WS;
  const int c0 = min(kc1, kc0 + wk * per), c1 = min(kc1, c0 + per);
  // with PP_UPSAMPLE2 (4-byte staging only) the conv's input is the nearest
  // x2 upsampling of x: a.h x a.w is the upsampled size and element (gy, gx)
  // is read from x[gy / 2][gx / 2]
  const bool up = !V4 && !BF && D == 1 && S == 1 && (a.flags & PP_UPSAMPLE2) != 0;
  const uint32_t sh = up ? a.h >> 1 : a.h, sw = up ? a.w >> 1 : a.w;   // stored input size
  const uint32_t chan_bytes = sh * sw * ES;
  const uint8_t* xi = static_cast<const uint8_t*>(a.x) + static_cast<size_t>(img) * a.c_in * sh * sw * ES;

  float* const ring = lds + wk * G::RING;
  const uint32_t ring_b = lds_addr(ring);
  constexpr uint32_t LW0 = 4u * G::PATCH;   // weights' byte offset in a ring slot

  // ---- per-lane staging offsets (bytes in one channel, + the DMA shift).
  // A load t of a lane stages the PE = 16 / ES (16-byte staging) or 4 / ES
  // (4-byte staging) elements PE (64 t + lane) .. + PE - 1 of the tile, all in
  // one tile row (LSTR is a multiple of PE) and all inside or all outside the
  // image (the row starts at a multiple of PE, w is a multiple of PE).  A
  // DMA's LDS bytes start at DPB t within the channel's slot.
  constexpr uint32_t PE = (V4 ? 16u : 4u) / ES;
  uint32_t qoff[NQ];
#pragma unroll
  for (int t = 0; t < NQ; ++t) {
    const uint32_t e = PE * (64u * t + lane);
    const uint32_t row = e / LSTR, col = e % LSTR;
    const uint32_t gy = static_cast<uint32_t>(iy0 + static_cast<int>(row));
    const uint32_t gx = static_cast<uint32_t>(ixa + static_cast<int>(col));
    const bool ok = e < static_cast<uint32_t>(G::AREA) && gy < a.h && gx < a.w;
    const uint32_t el = up ? (gy >> 1) * sw + (gx >> 1) : gy * a.w + gx;
    qoff[t] = ok ? el * ES + kDmaShift - ((static_cast<uint32_t>(G::DPB) * t) & 4095u) : 0x80000000u;
  }

  const uint8_t* blob = a.blob;
  const u32x4 brs = make_rsrc_below(blob, a.blob_bytes, kDmaShift);
  u32x4 cr = make_rsrc_below(xi + static_cast<size_t>(c0) * chan_bytes, chan_bytes, kDmaShift);
  // one channel's DMAs into ring slot sb (LDS byte address).  A channel past
  // the wave's range is staged all the same through descriptors of range 0
  // (every lane out of range: no memory is read, zeros land in a slot nobody
  // reads), so that the number of DMAs in flight never depends on where the
  // range ends and every wait below is one constant count.
  auto dma_patch = [&](uint32_t sb, bool live) __attribute__((always_inline)) {
    u32x4 d = cr;
    d.z = live ? cr.z : 0u;
    static_for<0, NQ>([&](auto ti) __attribute__((always_inline)) {
      constexpr int T = decltype(ti)::value;
      if constexpr (V4)
        dma_b128_at<1024u * T, 1024u * (T - 1), T == 0>(d, qoff[T], sb);
      else
        dma_b32_at<256u * T, 256u * (T - 1), T == 0>(d, qoff[T], sb);
    });
    cr = next_channel(cr, chan_bytes);
  };
  // expanded weights of a channel (its compact index: woff + 4 * rank of the
  // slot among the kept ones + tap).  fp32: lane j < 32 loads tap j % 4 of
  // slot j / 4; bf16: lane j < 16 loads the dword of taps 2 (j % 2), + 1 of
  // slot j / 2 (4-tap kernels: no padding, dword-aligned)
  constexpr uint32_t WPL = BF ? 2u : 1u;   // taps per lane
  const uint32_t wslot = static_cast<uint32_t>(lane) / (4u / WPL);
  const bool wlane = lane < static_cast<int>(32u / WPL);
  const uint32_t wlow = wlane ? (1u << wslot) - 1u : 0u;
  const uint32_t wbit = wlane ? 1u << wslot : 0u;
  const uint32_t wbase = a.off_w + 4u * (lane & (4 / WPL - 1)) + kDmaShift - (LW0 & 4095u);
  auto dma_weights = [&](uint32_t wo, uint32_t sb, bool live) __attribute__((always_inline)) {
    u32x4 d = brs;
    d.z = live ? brs.z : 0u;
    const uint32_t kept = wo >> 24;
    const uint32_t o = wbase + ES * ((wo & 0xFFFFFFu) + 4u * __builtin_popcount(kept & wlow));
    dma_b32_at<LW0, static_cast<uint32_t>(G::DPB) * (NQ - 1), false>(d, (kept & wbit) ? o : 0x80000000u, sb);
  };

  // metadata: woff word (weight offset | kept-slot mask << 24) and the 8
  // pattern codes of (group, channel), read by scalar loads at byte offsets
  // that move on by one entry per channel.  Reads for channels past the
  // layer's last (at most NS entries past the end of the woff array, one
  // past the end of the codes) land in the sections that follow them in the
  // blob (woff, weights, bias: the blob validation enforces that order) and
  // feed only the staging of channels nobody reads.
  uint32_t wo_at = a.off_woff + 4u * (grp * a.c_in + c0);
  uint32_t cd_at = a.off_codes + 8u * (grp * a.c_in + c0);

  // the slot group's output channels and biases for the epilogue, lane s <
  // 8 holding slot s's (loaded before the first DMA: in-order completion
  // keeps the DMA wait counts below valid)
  const uint32_t pslot = grp * 8 + (lane & 7);
  const uint32_t perm_l = *reinterpret_cast<const uint32_t*>(blob + a.off_perm + 4u * pslot);
  const float bias_l = *reinterpret_cast<const float*>(blob + a.off_bias + 4u * pslot);
  __builtin_amdgcn_sched_barrier(0);

  float acc[8][R][CC];
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int qq = 0; qq < CC; ++qq) acc[s][r][qq] = 0.0f;
  if (c0 < c1) {
    constexpr int QV = NQ + (PW ? 0 : 1);   // DMAs per lane and channel
    constexpr int DPF = NS - 1;  // channels DMA'd ahead
    constexpr uint32_t SLOTB = 4u * SLOT;
    // ring slots (LDS byte addresses): rd holds channel c, and channel c +
    // DPF goes to the slot channel c - 1 used (its reads are done by then)
    const uint32_t ring_end = ring_b + NS * SLOTB;
    uint32_t rd = ring_b;
    uint32_t wr = ring_b + DPF * SLOTB;
    // prologue: channel c0's halo before anything else, then channels up
    // to c0 + DPF - 1
    dma_patch(ring_b, true);
    __builtin_amdgcn_sched_barrier(0);
    uint32_t wo_pre[DPF + 1];
#pragma unroll
    for (int i = 0; i <= DPF; ++i) wo_pre[i] = kern::sload<uint32_t>(blob, wo_at + 4u * i);
    uint2 code_c = kern::sload<uint2>(blob, cd_at);
    // PW: the prepared weights of (group, channel) e at byte 128 e
    const uint32_t wp_at0 = 128u * (grp * a.c_in);
    float4 wsc[8];
    if constexpr (PW) {
#pragma unroll
      for (int s = 0; s < 8; ++s) wsc[s] = kern::sload<float4>(a.wprep, wp_at0 + 128u * c0 + 16u * s);
    }
    wait_lgkm();
    if constexpr (!PW) dma_weights(wo_pre[0], ring_b, true);
#pragma unroll
    for (int i = 1; i < DPF; ++i) {
      const bool live = c0 + i < c1;
      dma_patch(ring_b + i * SLOTB, live);
      if constexpr (!PW) dma_weights(wo_pre[i], ring_b + i * SLOTB, live);
    }
    uint32_t kept_c = wo_pre[0] >> 24;
    uint32_t wo_n = wo_pre[DPF];   // woff word of channel c + DPF
    // the lane's patch in a slot: fp32 from element lx CC of its first row;
    // bf16 from the dword holding element lx CC + SH - 1 (read_row_bf)
    const uint32_t lane_b =
        BF ? ES * ((ly * R) * LSTR + lx * CC + G::SH - 1) : 4u * ((ly * R * S) * LSTR + lx * CC * S);

#pragma unroll 1
    for (int c = c0; c < c1; ++c) {
      // channel c has landed once the DMAs of the DPF - 1 channels after it
      // are the only ones in flight
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_waitcnt(vmcnt_imm((DPF - 1) * QV));
      asm volatile("" ::: "memory");
      // the patch and the expanded weights of slots 0-3 of channel c (those
      // of slots 4-7 are read into the same registers once slots 0-3 are
      // done: 16 fewer registers, which lets the 2 x 4 tilings hold four
      // waves per SIMD)
      const float* cur = ring + (rd - ring_b) / 4u;
      const float4* wc = reinterpret_cast<const float4*>(cur + G::PATCH);
      float w[4][4];
      uint32_t wq[16];   // bf16: the 8 slots' taps as pairs
      float p[PR][PC];
      {
        if constexpr (BF) {
          if constexpr (!PW) {
            const uint4* wu = reinterpret_cast<const uint4*>(cur + G::PATCH);
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const uint4 v = wu[k];
              wq[4 * k] = v.x; wq[4 * k + 1] = v.y; wq[4 * k + 2] = v.z; wq[4 * k + 3] = v.w;
            }
          }
          const uint8_t* pb = reinterpret_cast<const uint8_t*>(cur) + lane_b;
#pragma unroll
          for (int r = 0; r < PR; ++r) read_row_bf<PC, CC % 4 == 0>(p[r], pb + r * LSTR * ES);
        } else {
          if constexpr (!PW) {
#pragma unroll
            for (int s = 0; s < 4; ++s) {
              const float4 v = wc[s];
              w[s][0] = v.x; w[s][1] = v.y; w[s][2] = v.z; w[s][3] = v.w;
            }
          }
#pragma unroll
          for (int r = 0; r < PR; ++r)
            read_row<G::SH, G::SH, PC, G::VWL, false>(p[r], cur + lane_b / 4u + r * LSTR);
        }
      }
      // channel c's reads, and the scalar loads of the previous step
      wait_lgkm();
      __builtin_amdgcn_sched_barrier(0);
      // channel c + DPF into the slot channel c - 1 used (its reads are done)
      {
        const bool live = c + DPF < c1;
        dma_patch(wr, live);
        if constexpr (!PW) dma_weights(wo_n, wr, live);
      }
      // metadata for the next step: waited for there, while this channel's
      // FMAs run
      wo_at += 4u;
      cd_at += 8u;
      const uint32_t wo_nn = kern::sload<uint32_t>(blob, wo_at + 4u * DPF);
      const uint32_t wo_c1 = kern::sload<uint32_t>(blob, wo_at);
      const uint2 code_c1 = kern::sload<uint2>(blob, cd_at);
      uint32_t warm0 = 0, warm1 = 0;
      if constexpr (PW) {
        // the weights of two channels ahead brought into the scalar cache
        // (one dword of each of their two 64-byte lines), so that the loads
        // of the next channel at the end of this step hit it
        const uint32_t cw = c + 2 < c1 ? c + 2 : c1 - 1;
        warm0 = kern::sload<uint32_t>(a.wprep, wp_at0 + 128u * cw);
        warm1 = kern::sload<uint32_t>(a.wprep, wp_at0 + 128u * cw + 64u);
      }
      __builtin_amdgcn_sched_barrier(0);
      const uint32_t kept = kept_c;
      uint32_t kc = kept;
      asm volatile("" : "+s"(kc));   // fresh slot tests
      {
        const uint32_t cx = code_c.x, cy = code_c.y;
        if constexpr (PW) {
          (void)w;
          (void)wq;
          static_for<0, 8>([&](auto si) __attribute__((always_inline)) {
            constexpr int s = decltype(si)::value;
            if (!((kc >> s) & 1u)) return;
            // the slot's 4 weights into VGPRs (an SGPR operand would halve the FMA rate)
            float w0, w1, w2, w3;
            asm volatile("v_mov_b32 %0, %4\n v_mov_b32 %1, %5\n v_mov_b32 %2, %6\n v_mov_b32 %3, %7"
                         : "=v"(w0), "=v"(w1), "=v"(w2), "=v"(w3)
                         : "s"(wsc[s].x), "s"(wsc[s].y), "s"(wsc[s].z), "s"(wsc[s].w));
            apply_canon8_bits<8 * (s & 3), S, D>(s < 4 ? cx : cy, acc[s], p, w0, w1, w2, w3);
          });
        } else if constexpr (BF) {
          // a kept slot's 4 taps widened from its two dwords
          static_for<0, 8>([&](auto si) __attribute__((always_inline)) {
            constexpr int s = decltype(si)::value;
            if (!((kc >> s) & 1u)) return;
            const uint32_t u0 = wq[2 * s], u1 = wq[2 * s + 1];
            apply_canon8_bits<8 * (s & 3), S, D>(s < 4 ? cx : cy, acc[s], p, bf_lo(u0), bf_hi(u0), bf_lo(u1), bf_hi(u1));
          });
        } else {
          static_for<0, 4>([&](auto si) __attribute__((always_inline)) {
            constexpr int s = decltype(si)::value;
            if (!((kc >> s) & 1u)) return;
            apply_canon8_bits<8 * s, S, D>(cx, acc[s], p, w[s][0], w[s][1], w[s][2], w[s][3]);
          });
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            const float4 v = wc[4 + s];
            w[s][0] = v.x; w[s][1] = v.y; w[s][2] = v.z; w[s][3] = v.w;
          }
          static_for<4, 8>([&](auto si) __attribute__((always_inline)) {
            constexpr int s = decltype(si)::value;
            if (!((kc >> s) & 1u)) return;
            apply_canon8_bits<8 * (s - 4), S, D>(cy, acc[s], p, w[s - 4][0], w[s - 4][1], w[s - 4][2], w[s - 4][3]);
          });
        }
      }
      kept_c = wo_c1 >> 24;
      code_c = code_c1;
      wo_n = wo_nn;
      if constexpr (PW) {
        asm volatile("" ::"s"(warm0), "s"(warm1));
        // the next channel's weights (the last channel reloads its own:
        // nothing past the wave's range is read), waited for with the next
        // step's LDS reads
        const uint32_t cn = c + 1 < c1 ? c + 1 : c;
#pragma unroll
        for (int s = 0; s < 8; ++s) wsc[s] = kern::sload<float4>(a.wprep, wp_at0 + 128u * cn + 16u * s);
      }
      wr = rd;
      rd = rd + SLOTB == ring_end ? ring_b : rd + SLOTB;
        }
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));   // no DMA may land in the exchange area below
  }

  // ---- epilogue
  const bool pool = (a.flags & PP_MAXPOOL2) != 0;
  const bool relu = (a.flags & PP_RELU) != 0;
  const bool split = a.ksplit > 1;
  // PP_ACCUMULATE: y holds a residual r and becomes r + act(conv + bias);
  // PP_PIXSHUF2: output channel o is stored to channel o / 4 of the 2 ho x
  // 2 wo output, row 2 oy + bit 1 of o, column 2 ox + bit 0 of o
  const bool accum = (a.flags & PP_ACCUMULATE) != 0;
  const bool shuf = (a.flags & PP_PIXSHUF2) != 0;
  const uint32_t pho = a.ho / 2, pwo = a.wo / 2;
  const size_t yoff = static_cast<size_t>(img) * a.c_out * (pool ? pho * pwo : a.ho * a.wo);
  float* __restrict__ y = static_cast<float*>(a.y) + yoff;
  uint16_t* __restrict__ yb = static_cast<uint16_t*>(a.y) + yoff;   // bf16 output
  const int oxl = ox0 + lx * CC;
  const bool vec = (CC % 4 == 0) && (a.wo % 4 == 0);
  // a row r of slot s: finish (bias, activation, store through perm) or,
  // under a channel split, store the partial sums to this split's block
  constexpr int BLK = 8 * R * CC * 64;
  const uint32_t item = ((img * a.tiles_y.d + ty) * a.tiles_x.d + tx) * a.groups.d + grp;
  auto finish = [&](int s, int r, float (&v)[CC]) __attribute__((always_inline)) {
    if (split) {
      float* pb = a.part + static_cast<size_t>(item * a.ksplit + ks) * BLK + lane;
#pragma unroll
      for (int qq = 0; qq < CC; ++qq) pb[((s * R + r) * CC + qq) * 64] = v[qq];
      return;
    }
    const uint32_t o = __builtin_amdgcn_readlane(perm_l, s);
    const float bias = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(uint32_t, bias_l), s));
    if (o >= a.c_out) return;   // padding slot
    const int oy = oy0 + ly * R + r;
    if (oy >= static_cast<int>(a.ho)) return;
#pragma unroll
    for (int qq = 0; qq < CC; ++qq) {
      v[qq] += bias;
      if (relu) v[qq] = fmaxf(v[qq], 0.0f);
    }
    if constexpr (BF) {
      // one rounding to bf16 (PP_ACCUMULATE: the stored residual plus the
      // rounded activated value, rounded again); CC (even) outputs as dword
      // pairs when the row and the lane's first column are even
      uint16_t* row = yb + (static_cast<size_t>(o) * a.ho + oy) * a.wo;
      if (a.wo % 2 == 0 && oxl + CC <= static_cast<int>(a.wo)) {
#pragma unroll
        for (int qq = 0; qq < CC; qq += 2) {
          uint32_t* pr = reinterpret_cast<uint32_t*>(row + oxl + qq);
          uint32_t lo = bf_rne(v[qq]), hi = bf_rne(v[qq + 1]);
          if (accum) {
            const uint32_t old = *pr;
            lo = bf_rne(bf_lo(old) + bf_lo(lo));
            hi = bf_rne(bf_hi(old) + bf_lo(hi));
          }
          *pr = lo | (hi << 16);
        }
      } else {
#pragma unroll
        for (int qq = 0; qq < CC; ++qq)
          if (oxl + qq < static_cast<int>(a.wo)) {
            uint32_t b = bf_rne(v[qq]);
            if (accum) b = bf_rne(bf_lo(row[oxl + qq]) + bf_lo(b));
            row[oxl + qq] = static_cast<uint16_t>(b);
          }
      }
      return;
    }
    if (shuf) {
      float* row2 = y + (static_cast<size_t>(o >> 2) * 2 * a.ho + 2 * oy + ((o >> 1) & 1)) * 2 * a.wo + (o & 1);
#pragma unroll
      for (int qq = 0; qq < CC; ++qq)
        if (oxl + qq < static_cast<int>(a.wo)) row2[2 * (oxl + qq)] = v[qq];
      return;
    }
    float* row = y + (static_cast<size_t>(o) * a.ho + oy) * a.wo;
    if (vec && oxl + CC <= static_cast<int>(a.wo)) {
#pragma unroll
      for (int qq = 0; qq < CC; qq += 4) {
        float4* pr = reinterpret_cast<float4*>(row + oxl + qq);
        float4 t = make_float4(v[qq], v[qq + 1], v[qq + 2], v[qq + 3]);
        if (accum) {
          const float4 old = *pr;
          t = make_float4(old.x + t.x, old.y + t.y, old.z + t.z, old.w + t.w);
        }
        *pr = t;
      }
    } else {
#pragma unroll
      for (int qq = 0; qq < CC; ++qq)
        if (oxl + qq < static_cast<int>(a.wo)) row[oxl + qq] = accum ? row[oxl + qq] + v[qq] : v[qq];
    }
  };
  // rows r, r + 1 of slot s, 2 x 2 max pooled (windows wholly inside the
  // output; floor), the max taken over the activated values
  auto finish_pool = [&](int s, int r, float (&v0)[CC], float (&v1)[CC]) __attribute__((always_inline)) {
    const uint32_t o = __builtin_amdgcn_readlane(perm_l, s);
    const float bias = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(uint32_t, bias_l), s));
    if (o >= a.c_out) return;
    const int oy = oy0 + ly * R + r;
    if (oy + 1 >= static_cast<int>(a.ho)) return;
    float* row = y + (static_cast<size_t>(o) * pho + oy / 2) * pwo;
    float m[CC / 2];
#pragma unroll
    for (int j = 0; j < CC / 2; ++j) {
      float t0 = v0[2 * j] + bias, t1 = v0[2 * j + 1] + bias, t2 = v1[2 * j] + bias, t3 = v1[2 * j + 1] + bias;
      if (relu) {
        t0 = fmaxf(t0, 0.0f); t1 = fmaxf(t1, 0.0f); t2 = fmaxf(t2, 0.0f); t3 = fmaxf(t3, 0.0f);
      }
      m[j] = fmaxf(fmaxf(t0, t1), fmaxf(t2, t3));
    }
    if constexpr (BF) {
      uint16_t* rowb = yb + (static_cast<size_t>(o) * pho + oy / 2) * pwo;
#pragma unroll
      for (int j = 0; j < CC / 2; ++j)
        if (oxl + 2 * j + 1 < static_cast<int>(a.wo)) rowb[oxl / 2 + j] = static_cast<uint16_t>(bf_rne(m[j]));
      return;
    }
#pragma unroll
    for (int j = 0; j < CC / 2; ++j)
      if (oxl + 2 * j + 1 < static_cast<int>(a.wo)) row[oxl / 2 + j] = m[j];
  };

  if constexpr (WS == 1) {
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      if constexpr (R % 2 == 0 && CC % 2 == 0) {
        if (pool && !split) {
#pragma unroll
          for (int r = 0; r < R; r += 2) finish_pool(s, r, acc[s][r], acc[s][r + 1]);
          continue;
        }
      }
#pragma unroll
      for (int r = 0; r < R; ++r) finish(s, r, acc[s][r]);
    }
  } else {
    // SPP slots per pass: every wave writes its partial rows, then unit u =
    // (slot of the pass, row or row pair) is summed over the WS waves in
    // wave order by wave u % WS
    constexpr int SPP = G::SPP;
#pragma unroll
    for (int s0 = 0; s0 < 8; s0 += SPP) {
      __syncthreads();
      {
        float* dst = lds + wk * SPP * G::XPS + lane;
#pragma unroll
        for (int ps = 0; ps < SPP; ++ps)
#pragma unroll
          for (int r = 0; r < R; ++r)
#pragma unroll
            for (int qq = 0; qq < CC; ++qq) dst[((ps * R + r) * CC + qq) * 64] = acc[s0 + ps][r][qq];
      }
      __syncthreads();
      auto gather = [&](int ps, int r, float (&v)[CC]) __attribute__((always_inline)) {
#pragma unroll
        for (int qq = 0; qq < CC; ++qq) {
          float t = 0.0f;
#pragma unroll
          for (int k = 0; k < WS; ++k) t += lds[k * SPP * G::XPS + ((ps * R + r) * CC + qq) * 64 + lane];
          v[qq] = t;
        }
      };
      bool pooled = false;
      if constexpr (R % 2 == 0 && CC % 2 == 0) {
        if (pool && !split) {
          pooled = true;
          constexpr int NUP = SPP * (R / 2);
          for (int u = wk; u < NUP; u += WS) {
            const int ps = u / (R / 2), r = 2 * (u % (R / 2));
            float v0[CC], v1[CC];
            gather(ps, r, v0);
            gather(ps, r + 1, v1);
            finish_pool(s0 + ps, r, v0, v1);
          }
        }
      }
      if (!pooled) {
        constexpr int NU = SPP * R;
        for (int u = wk; u < NU; u += WS) {
          const int ps = u / R, r = u % R;
          float v[CC];
          gather(ps, r, v);
          finish(s0 + ps, r, v);
        }
      }
    }
  }
}

// Second pass of a channel split: y = act(sum over the ksplit partial-sum
// blocks of a tile, in split order, + bias), stored through perm; with
// PP_MAXPOOL2 the 2 x 2 max of the activated sums (windows wholly inside the
// output).  One workgroup per (image, tile, slot group).  A thread first
// works out where each of its outputs (or pooled windows) sits in a partial
// block, then issues the loads of one split for all of them at once, so the
// pass costs about one memory round trip per split, not one per output.
template <int R, int CC, int LW, bool BF = false>
__global__ __launch_bounds__(256) void pp_lean_reduce_kernel(LeanParams a) {
  constexpr int LH = 64 / LW, TH = LH * R, TW = LW * CC;
  constexpr int BLK = 8 * R * CC * 64;
  const uint32_t item = blockIdx.x;
  uint32_t t = fdiv(item, a.groups);
  const uint32_t grp = item - t * a.groups.d;
  uint32_t t2 = fdiv(t, a.tiles_x);
  const uint32_t tx = t - t2 * a.tiles_x.d;
  t = fdiv(t2, a.tiles_y);
  const uint32_t ty = t2 - t * a.tiles_y.d;
  const uint32_t img = t;
  const float* pb = a.part + static_cast<size_t>(item) * a.ksplit * BLK;
  const bool relu = (a.flags & PP_RELU) != 0;
  uint32_t perm[8];
  float biasv[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    perm[s] = sload<uint32_t>(a.blob, a.off_perm + 4u * (grp * 8u + s));
    biasv[s] = sload<float>(a.blob, a.off_bias + 4u * (grp * 8u + s));
  }
  // offset of output (s, yl, xl) of the tile in a partial block
  auto at = [](int s, int yl, int xl) {
    return ((s * R + yl % R) * CC + xl % CC) * 64 + (yl / R) * LW + xl / CC;
  };
  auto act = [&](float v, int s) {
    v += biasv[s];
    return relu ? fmaxf(v, 0.0f) : v;
  };
  if (a.flags & PP_MAXPOOL2) {
    const uint32_t pho = a.ho / 2, pwo = a.wo / 2;
    const size_t ypo = static_cast<size_t>(img) * a.c_out * pho * pwo;
    constexpr int PH = TH / 2, PW = TW / 2, NW = 8 * PH * PW, PER = (NW + 255) / 256;
    int off[PER][4];
    float v[PER][4];
#pragma unroll
    for (int m = 0; m < PER; ++m) {
      const int i = min(static_cast<int>(threadIdx.x) + 256 * m, NW - 1);
      const int s = i / (PH * PW), px = i % PW, py = (i / PW) % PH;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        off[m][j] = at(s, 2 * py + (j >> 1), 2 * px + (j & 1));
        v[m][j] = 0.0f;
      }
    }
    for (uint32_t k = 0; k < a.ksplit; ++k) {
      const float* pk = pb + static_cast<size_t>(k) * BLK;
#pragma unroll
      for (int m = 0; m < PER; ++m)
#pragma unroll
        for (int j = 0; j < 4; ++j) v[m][j] += pk[off[m][j]];
    }
#pragma unroll
    for (int m = 0; m < PER; ++m) {
      const int i = static_cast<int>(threadIdx.x) + 256 * m;
      if (i >= NW) continue;
      const int s = i / (PH * PW), px = i % PW, py = (i / PW) % PH;
      const uint32_t oy = ty * TH + 2 * py, ox = tx * TW + 2 * px;
      if (oy + 1 >= a.ho || ox + 1 >= a.wo) continue;
      const uint32_t o = perm[s];
      if (o >= a.c_out) continue;
      const float r = fmaxf(fmaxf(act(v[m][0], s), act(v[m][1], s)), fmaxf(act(v[m][2], s), act(v[m][3], s)));
      const size_t at_p = ypo + (static_cast<size_t>(o) * pho + oy / 2) * pwo + ox / 2;
      if constexpr (BF)
        static_cast<uint16_t*>(a.y)[at_p] = static_cast<uint16_t>(bf_rne(r));
      else
        static_cast<float*>(a.y)[at_p] = r;
    }
    return;
  }
  const size_t yo = static_cast<size_t>(img) * a.c_out * a.ho * a.wo;
  constexpr int NO = 8 * TH * TW, PER = (NO + 255) / 256;
  int off[PER];
  float v[PER];
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    const int i = min(static_cast<int>(threadIdx.x) + 256 * m, NO - 1);
    const int s = i / (TH * TW), xl = i % TW, yl = (i / TW) % TH;
    off[m] = at(s, yl, xl);
    v[m] = 0.0f;
  }
  for (uint32_t k = 0; k < a.ksplit; ++k) {
    const float* pk = pb + static_cast<size_t>(k) * BLK;
#pragma unroll
    for (int m = 0; m < PER; ++m) v[m] += pk[off[m]];
  }
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    const int i = static_cast<int>(threadIdx.x) + 256 * m;
    if (i >= NO) continue;
    const int s = i / (TH * TW), xl = i % TW, yl = (i / TW) % TH;
    const uint32_t oy = ty * TH + yl, ox = tx * TW + xl;
    if (oy >= a.ho || ox >= a.wo) continue;
    const uint32_t o = perm[s];
    if (o >= a.c_out) continue;
    const size_t at_y = (a.flags & PP_PIXSHUF2)
                            ? (static_cast<size_t>(o >> 2) * 2 * a.ho + 2 * oy + ((o >> 1) & 1)) * 2 * a.wo + 2 * ox + (o & 1)
                            : (static_cast<size_t>(o) * a.ho + oy) * a.wo + ox;
    const float r = act(v[m], s);
    if constexpr (BF) {
      // (no shuffle in bf16; accumulate as in the first pass)
      uint16_t* y = static_cast<uint16_t*>(a.y) + yo;
      uint32_t b = bf_rne(r);
      if (a.flags & PP_ACCUMULATE) b = bf_rne(bf_lo(y[at_y]) + bf_lo(b));
      y[at_y] = static_cast<uint16_t>(b);
    } else {
      float* y = static_cast<float*>(a.y) + yo;
      y[at_y] = (a.flags & PP_ACCUMULATE) ? y[at_y] + r : r;
    }
  }
}

#ifndef __HIPCC_RTC__   // host side
template <int R, int CC, int LW, int WS, bool V4, bool BF = false, bool PW = false, int D = 1, int S = 1>
hipError_t launch_lean_tiling(LeanParams p, int n, hipStream_t st) {
  using G = LGeo<R, CC, LW, WS, V4, BF, D, S>;
  if constexpr (!G::fits) {
    return hipErrorInvalidConfiguration;
  } else {
    if (V4 && (p.w % (BF ? 8 : 4) != 0 || (p.flags & PP_UPSAMPLE2))) return hipErrorInvalidConfiguration;
    if (BF && (p.w % 2 != 0 || (p.flags & (PP_UPSAMPLE2 | PP_PIXSHUF2))))
      return hipErrorInvalidConfiguration;
    if ((D != 1 || S != 1) && (p.flags & PP_UPSAMPLE2)) return hipErrorInvalidConfiguration;
    const uint32_t tx = (p.wo + G::TW - 1) / G::TW, ty = (p.ho + G::TH - 1) / G::TH;
    const uint32_t ng = p.groups.d;
    if (p.ksplit < 1 || p.ksplit > p.c_in || (p.ksplit > 1 && !p.part)) return hipErrorInvalidValue;
    if (static_cast<uint64_t>(p.ksplit) * p.c_in >= (1ull << 31)) return hipErrorInvalidValue;   // fdiv range
    p.tiles_x = make_fastdiv(tx);
    p.tiles_y = make_fastdiv(ty);
    p.splits = make_fastdiv(p.ksplit);
    const size_t nb = static_cast<size_t>(ng) * p.ksplit * tx * ty * n;
    if (nb == 0 || nb > 0x7FFFFFFFull) return hipErrorInvalidConfiguration;
    if (PW && !p.wprep) return hipErrorInvalidValue;
    hipLaunchKernelGGL((pp_conv3x3_lean_kernel<R, CC, LW, WS, V4, BF, PW, D, S>), dim3(static_cast<uint32_t>(nb)),
                       dim3(WS * 64), 0, st, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.ksplit == 1) return e;
    hipLaunchKernelGGL((pp_lean_reduce_kernel<R, CC, LW, BF>), dim3(static_cast<uint32_t>(nb / p.ksplit)), dim3(256), 0,
                       st, p);
    return hipGetLastError();
  }
}
#endif

}  // namespace kern

#ifndef __HIPCC_RTC__
// the dilation-2 tilings (conv_pp_lean_d2.hip) and the stride-2 ones
// (conv_pp_lean_s2.hip): launch, and LDS bytes (0: not built for that case,
// or does not fit)
hipError_t launch_lean_d2(int id, const LeanParams& p, int n, bool pw, hipStream_t st);
long lean_lds_bytes_d2(int id);
hipError_t launch_lean_s2(int id, const LeanParams& p, int n, bool pw, hipStream_t st);
long lean_lds_bytes_s2(int id);
#endif
}  // namespace pp
