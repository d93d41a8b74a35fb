// conv_pp_wave.hpp -- pattern/connectivity-pruned 3x3 convolution for the
// canonical 8-pattern library, "wave pipeline" form (gfx950).
//
// Same result as pp_conv3x3_kernel (pattern + connectivity pruning, Sec. 2;
// compact storage and filter reorder, Sec. 3; conv fused with bias and
// activation, Sec. 3), organised so that a wave never waits on another wave
// while it walks its input channels:
//
//   * A workgroup owns one output tile of one image and ONE slot group (8
//     packed filters).  Its WS waves split the input channels into WS
//     contiguous ranges; each wave runs its range on its own and the partial
//     sums are combined at the end through LDS in a fixed order
//     (deterministic).
//   * Lanes are output pixels (R x CC outputs per lane, LW lanes across), as
//     in the other kernel, so the pattern of a (slot, channel) kernel is
//     wave-uniform and selects a code path whose tap offsets are compile-time
//     constants.
//   * Per wave, a software pipeline over its channels with a private 2-slot
//     LDS ring:  the halo tile of channel c+2 and the expanded weights of its
//     8 slots are loaded from global memory into registers while channel c is
//     computed; they are written to the LDS ring one channel later; the
//     channel's metadata (kept-slot mask, weight offset, pattern codes) comes
//     by scalar loads three channels ahead.  Within a channel, the patch and
//     the kept slots' weights are read from LDS together and waited for once.
//   * The halo tile is read with 16-byte loads when the image width is a
//     multiple of 4 (the tile origin is moved down to a multiple of 4 columns
//     and the patch reads are shifted back), else element by element;
//     out-of-image elements read zero through the buffer range check.
#pragma once

#include "conv_pp_kernel.hpp"

namespace pp {
namespace kern {

template <int LIB, int S, int D, int R, int CC, int LW, int WS, bool ABF, bool PIPE_REQ>
struct WGeo {
  // expanded weights per slot in LDS: 4 taps (canonical library) or the 9
  // taps padded to 12 (all-ones library)
  static constexpr int KW = LIB == kLibDense9 ? 12 : 4;
  static constexpr int KT = LIB == kLibDense9 ? 9 : 4;     // taps per kept kernel
  static constexpr int WAREA = (8 * KW + 63) / 64 * 64;
  static constexpr int NWL = WAREA / 64;                   // weight loads per lane
  static constexpr int LH = 64 / LW;
  static constexpr int TH = LH * R, TW = LW * CC;          // output tile
  static constexpr int PR = (R - 1) * S + 2 * D + 1;       // patch rows
  static constexpr int PC = (CC - 1) * S + 2 * D + 1;      // patch cols
  static constexpr int TIH = (TH - 1) * S + 2 * D + 1;     // input tile rows
  static constexpr int TIW = (TW - 1) * S + 2 * D + 1;     // input tile cols
  // + up to 3 columns in front of the tile when its origin is moved down to a
  // multiple of 4
  static constexpr int LSTR = wave_row_stride((TIW + 3 + 3) / 4 * 4, R * S);
  static constexpr int AREA = TIH * LSTR;
  static constexpr int NQ = (AREA + 255) / 256;           // 4-float staging groups per lane
  static constexpr int PATCH = NQ * 256;                  // floats per staged channel
  static constexpr int SLOT = PATCH + WAREA;
  // ring slots per wave: fp32 channels are DMA'd straight into LDS DPF
  // channels ahead (DPF + 1 slots); bf16 goes through registers (2 slots)
  static constexpr int NSLOT = wave_nslot(R, CC, LW, WS, S, D, WAREA, ABF);
  static constexpr int DPF = NSLOT - 1;
  static_assert(SLOT == wave_slot_floats(R, CC, LW, S, D, WAREA), "planner and kernel disagree on the slot size");
  static constexpr int RING = NSLOT * SLOT;               // per wave
  static constexpr int NACC = 8 * R * CC;
  // fp32 canonical library, on request: the next channel's patch and weights
  // are read into a second register set while this one is computed (both
  // sets and the accumulators must fit the registers a wave may hold: 256,
  // or 128 with 16 waves per workgroup)
  static constexpr int VBUDGET = WS > 8 ? 128 : 256;
  static constexpr bool PIPE = PIPE_REQ && !ABF && LIB == kLibCanon8 && NACC + 2 * (PR * PC + 8 * KW) + 24 <= VBUDGET;
  // partial-sum exchange: PS slots at a time, every wave writes PS*R*CC floats per lane
  static constexpr int PS = 2;
  static constexpr int XCH = WS * PS * R * CC * 64;
  static constexpr int LDS_FLOATS = (WS * RING > XCH) ? WS * RING : XCH;
  static_assert(LDS_FLOATS == wave_lds_floats(R, CC, LW, WS, S, D, WAREA, ABF),
                "planner and kernel disagree on LDS size");
  static constexpr bool fits = LDS_FLOATS * 4 <= 160 * 1024 && LW * LH == 64 && WS >= 1 && WS <= 16;
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// The DMA helpers below write and read M0, which the compiler treats as
// reserved; no code generated for these kernels keeps or sets a value in M0
// (no indirect register indexing), so M0 holds between set_m0 and the DMAs.
// They are inline assembly so that the compiler neither waits for the DMAs
// (the caller counts vmcnt) nor moves LDS reads across them.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"

// raw buffer descriptor (gfx9 layout: 48-bit base, stride 0, num_records
// bytes, 32-bit data format) as four SGPRs; offsets >= bytes read zero
__device__ __forceinline__ u32x4 make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  u32x4 r;
  r.x = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b));
  r.y = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b >> 32) & 0xFFFFu);
  r.z = __builtin_amdgcn_readfirstlane(bytes);
  r.w = 0x00020000u;
  return r;
}

// M0 for the LDS DMAs that follow (with the wait state the hardware needs
// between an M0 write and its use)
__device__ __forceinline__ void set_m0(uint32_t v) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0" :: "s"(v) : "memory", "m0");
}
// The descriptor is wave-uniform.  The run-time compiler can be an older
// one (a host process may have loaded its own copy first) that does not
// always prove it and then hands the asm VGPRs; a descriptor rebuilt from
// read-first-lanes keeps it in SGPRs.  A VMEM instruction needs 5 wait states
// after a VALU write of its SGPRs, and the compiler does not see that the
// asm is one, so the asm waits itself (PP_DMA_WAIT).
#ifdef __HIPCC_RTC__
#define PP_DMA_WAIT "s_nop 4\n\t"
#else
#define PP_DMA_WAIT ""
#endif
__device__ __forceinline__ u32x4 uniform_rsrc(u32x4 r) {
#ifdef __HIPCC_RTC__
  u32x4 u;
  u.x = __builtin_amdgcn_readfirstlane(r.x);
  u.y = __builtin_amdgcn_readfirstlane(r.y);
  u.z = __builtin_amdgcn_readfirstlane(r.z);
  u.w = __builtin_amdgcn_readfirstlane(r.w);
  return u;
#else
  return r;
#endif
}
// global -> LDS DMA of 16 (4) bytes per lane with immediate offset OFF: it
// moves both the global offset and the LDS address, so lane l's data lands
// at LDS byte M0 + OFF + 16 l (4 l) and comes from offset voff + OFF
template <uint32_t OFF>
__device__ __forceinline__ void dma_lds_b128_at(u32x4 rsrc, uint32_t voff) {
  asm volatile(PP_DMA_WAIT "buffer_load_dwordx4 %0, %1, 0 offen offset:%2 lds" :: "v"(voff), "s"(uniform_rsrc(rsrc)),
               "n"(OFF) : "memory");
}
template <uint32_t OFF>
__device__ __forceinline__ void dma_lds_b32_at(u32x4 rsrc, uint32_t voff) {
  asm volatile(PP_DMA_WAIT "buffer_load_dword %0, %1, 0 offen offset:%2 lds" :: "v"(voff), "s"(uniform_rsrc(rsrc)),
               "n"(OFF) : "memory");
}

#pragma clang diagnostic pop

// A channel's DMAs land at LDS byte offsets L from its ring slot; each is
// issued with immediate offset L % 4096 and M0 = slot + (L - L % 4096), set
// once per 4 KB group.  The descriptors' bases sit kDmaShift bytes below the
// data (ranges kDmaShift bytes longer), and every in-range per-lane offset
// carries + kDmaShift - L % 4096, so the offsets stay non-negative.
constexpr uint32_t kDmaShift = 4096;
template <uint32_t L, uint32_t LPREV, bool FIRST>
__device__ __forceinline__ void dma_b128_at(u32x4 rsrc, uint32_t voff, uint32_t slot) {
  if constexpr (FIRST || (L & ~4095u) != (LPREV & ~4095u)) set_m0(slot + (L & ~4095u));
  dma_lds_b128_at<(L & 4095u)>(rsrc, voff);
}
template <uint32_t L, uint32_t LPREV, bool FIRST>
__device__ __forceinline__ void dma_b32_at(u32x4 rsrc, uint32_t voff, uint32_t slot) {
  if constexpr (FIRST || (L & ~4095u) != (LPREV & ~4095u)) set_m0(slot + (L & ~4095u));
  dma_lds_b32_at<(L & 4095u)>(rsrc, voff);
}
template <int I, int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// a descriptor whose base sits `shift` bytes below `base` and whose range
// covers those bytes too (no access ever lands below base)
__device__ __forceinline__ u32x4 make_rsrc_below(const void* base, uint32_t bytes, uint32_t shift) {
  const uint64_t b = reinterpret_cast<uint64_t>(base) - shift;
  u32x4 r;
  r.x = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b));
  r.y = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(b >> 32) & 0xFFFFu);
  r.z = __builtin_amdgcn_readfirstlane(bytes + shift);
  r.w = 0x00020000u;
  return r;
}

// the same descriptor moved on by one channel of `bytes` bytes
__device__ __forceinline__ u32x4 next_channel(u32x4 r, uint32_t bytes) {
  const uint64_t b = (static_cast<uint64_t>(r.y) << 32 | r.x) + bytes;
  r.x = static_cast<uint32_t>(b);
  r.y = static_cast<uint32_t>(b >> 32) & 0xFFFFu;
  return r;
}

// s_waitcnt immediate that waits for vmcnt <= n (n <= 63) and nothing else
constexpr int vmcnt_imm(int n) {
  return (n > 63 ? 63 : n) < 0 ? 0x0F70 : (((n > 63 ? 63 : n) & 15) | (((n > 63 ? 63 : n) >> 4) << 14) | 0x0F70);
}

// one row of a lane's patch: elements [SH, SH + PC) of the staged row that
// starts at rb (rb aligned to VWL floats), read with the widest aligned LDS
// loads (a partly used pair at either end reads one extra element)
template <int J, int PC>
__device__ __forceinline__ void put_elem(float (&d)[PC], float v) {
  if constexpr (J >= 0 && J < PC) d[J] = v;
}
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
template <int I, int SH, int PC, int VWL, bool PIN>
__device__ __forceinline__ void read_row(float (&d)[PC], const float* rb) {
  constexpr int END = SH + PC;
  if constexpr (I < END) {
    if constexpr (VWL >= 4 && I % 4 == 0 && I + 4 <= END) {
      f32x4 v = *reinterpret_cast<const f32x4*>(__builtin_assume_aligned(rb + I, 16));
      if constexpr (PIN) asm("" : "+v"(v));   // keep the load whole (one aligned 16-byte read)
      put_elem<I - SH>(d, v.x);
      put_elem<I + 1 - SH>(d, v.y);
      put_elem<I + 2 - SH>(d, v.z);
      put_elem<I + 3 - SH>(d, v.w);
      read_row<I + 4, SH, PC, VWL, PIN>(d, rb);
    } else if constexpr (VWL >= 2 && !PIN && (I % 2 == 1 || I + 1 == END)) {
      // a single element of a pair: read it alone (a pair read whose other
      // half is dead lets the register allocator reuse that half for the
      // next read, which then has to wait for this one)
      put_elem<I - SH>(d, rb[I]);
      read_row<I + 1, SH, PC, VWL, PIN>(d, rb);
    } else if constexpr (VWL >= 2) {
      constexpr int B = I & ~1;
      f32x2 v = *reinterpret_cast<const f32x2*>(__builtin_assume_aligned(rb + B, 8));
      if constexpr (PIN) asm("" : "+v"(v));   // one aligned 8-byte read
      put_elem<B - SH>(d, v.x);
      put_elem<B + 1 - SH>(d, v.y);
      read_row<B + 2, SH, PC, VWL, PIN>(d, rb);
    } else {
      put_elem<I - SH>(d, rb[I]);
      read_row<I + 1, SH, PC, VWL, PIN>(d, rb);
    }
  }
}

// SH = (-pad) mod 4: the tile's first input column sits SH columns after a
// multiple of 4 (tile origins are multiples of 4 columns)
template <int LIB, int S, int D, int R, int CC, int LW, int WS, int SH, bool PIPE, class TA>
__global__ __launch_bounds__(WS * 64) void pp_conv3x3_wave_kernel(ConvParams a) {
  constexpr bool ABF = sizeof(TA) == 2;
  using G = WGeo<LIB, S, D, R, CC, LW, WS, ABF, PIPE>;
  constexpr int KW = G::KW, KT = G::KT, NWL = G::NWL;
  constexpr int PR = G::PR, PC = G::PC, LSTR = G::LSTR, NQ = G::NQ, SLOT = G::SLOT;
  static_assert(G::fits, "tiling does not fit");
  __shared__ __attribute__((aligned(16))) float lds[G::LDS_FLOATS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wk = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lx = lane % LW, ly = lane / LW;

  uint32_t blk = xcd_remap(blockIdx.x, gridDim.x);
  const int grp = blk % a.n_groups;
  blk /= a.n_groups;
  const int ks = blk % a.ksplit;       // this workgroup's share of the input channels
  blk /= a.ksplit;
  const int tx = blk % a.tiles_x;
  blk /= a.tiles_x;
  const int ty = blk % a.tiles_y;
  const int img = blk / a.tiles_y;

  const int oy0 = ty * G::TH, ox0 = tx * G::TW;
  const int iy0 = oy0 * S - a.pad, ix0 = ox0 * S - a.pad;
  // with PP_UPSAMPLE2 the conv's input is the nearest x2 upsampling of x:
  // a.h x a.w is the upsampled size and element (gy, gx) is read from
  // x[gy / 2][gx / 2] (element loads: a row of the tile is not contiguous)
  const bool up = (a.flags & PP_UPSAMPLE2) != 0;
  const int sh = up ? a.h >> 1 : a.h, sw = up ? a.w >> 1 : a.w;   // stored input size
  const bool v4 = !up && (a.w % 4) == 0;                // 16-byte (fp32) / 8-byte (bf16) row loads
  const int ixa = ix0 - SH;                             // a multiple of 4

  const TA* __restrict__ x = static_cast<const TA*>(a.x) + static_cast<size_t>(img) * a.c_in * sh * sw;
  const uint32_t chan_bytes = static_cast<uint32_t>(sh) * sw * sizeof(TA);
  const uint8_t* blob = a.blob;

  // ---- per-lane staging offsets (bytes within one channel), fixed for the
  // kernel.  Staged element e is tile row e / LSTR, column e % LSTR (global
  // column ixa + e % LSTR).  Load (t, j) of a lane stages element
  // e = 4*(64 t + lane) + j (16-byte loads, and every bf16 load), or
  // e = 64*(4 t + j) + lane (4-byte fp32 DMA, lane-contiguous in LDS).
  const bool lane4 = v4 || ABF;
  uint32_t qoff[NQ][4];
#pragma unroll
  for (int t = 0; t < NQ; ++t)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = lane4 ? 4 * (64 * t + lane) + j : 64 * (4 * t + j) + lane;
      const int row = e / LSTR, col = e % LSTR;
      const int gy = iy0 + row, gx = ixa + col;
      const bool ok = e < G::AREA && gy >= 0 && gy < a.h && gx >= 0 && gx < a.w;
      const uint32_t el = up ? static_cast<uint32_t>(gy >> 1) * sw + (gx >> 1) : static_cast<uint32_t>(gy) * a.w + gx;
      qoff[t][j] = ok ? el * static_cast<uint32_t>(sizeof(TA)) : 0x80000000u;
    }

  // ---- this wave's channel range
  // channels [kc0, kc1) of this workgroup (split ks of ksplit), then the
  // wave's contiguous part of them
  const int kc0 = static_cast<int>(static_cast<int64_t>(ks) * a.c_in / a.ksplit);
  const int kc1 = static_cast<int>(static_cast<int64_t>(ks + 1) * a.c_in / a.ksplit);
  const int per = (kc1 - kc0 + WS - 1) / WS;
  const int c0 = min(kc1, kc0 + wk * per), c1 = min(kc1, c0 + per);
  const uint32_t e_base = static_cast<uint32_t>(grp) * a.c_in;
  const uint32_t e_last = e_base + a.c_in - 1;

  float* const ring = lds + wk * G::RING;
  // a lane's patch row r starts SH elements after cur + lane_off + r*LSTR
  const int lane_off = (ly * R * S) * LSTR + lx * CC * S;
  constexpr int VWL = (CC * S) % 4 == 0 ? 4 : ((CC * S) % 2 == 0 ? 2 : 1);

  // metadata of channel c (clamped to the layer's last channel): woff word
  // and the 8 pattern codes, scalar loads
  struct Meta {
    uint32_t wo, cx, cy;
  };
  auto load_meta = [&](int c) __attribute__((always_inline)) {
    const uint32_t e = min(e_base + static_cast<uint32_t>(c), e_last);
    Meta m;
    m.wo = sload<uint32_t>(blob, a.off_woff + 4 * e);
    const uint2 cw = sload<uint2>(blob, a.off_codes + 8 * e);
    m.cx = cw.x;
    m.cy = cw.y;
    return m;
  };

  // staged data of one channel in registers
  float xs[NQ][4];
  float ws[NWL];
  const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(blob), static_cast<short>(0), static_cast<int>(a.blob_bytes), 0x00020000);

  // expanded weight e = 64 j + lane of a channel is tap e % KW of slot e / KW
  // (zero for padding taps, pruned slots and e >= 8 KW); its compact index is
  // woff + (stored weights per kernel) * rank(slot) + tap
  constexpr uint32_t KS = LIB == kLibDense9 ? (ABF ? 10u : 9u) : 4u;   // stored weights per kernel
  // per lane and weight load j: the slots below this lane's slot (rank mask),
  // its own slot bit (0 for padding taps and lanes past the 8 slots), its tap
  uint32_t wlow[NWL], wbit[NWL], wtp[NWL];
#pragma unroll
  for (int j = 0; j < NWL; ++j) {
    const int e = 64 * j + lane;
    const int s = e < 8 * KW ? e / KW : 8, t = e % KW;
    wlow[j] = s < 8 ? (1u << s) - 1u : 0u;
    wbit[j] = (s < 8 && t < KT) ? 1u << s : 0u;
    wtp[j] = static_cast<uint32_t>(t);
  }
  // adj: added to the in-range offsets (the DMA path's descriptor shift)
  auto weight_offs = [&](const Meta& m, uint32_t (&off)[NWL], auto adj) __attribute__((always_inline)) {
    const uint32_t kept = m.wo >> 24;
#pragma unroll
    for (int j = 0; j < NWL; ++j) {
      const uint32_t rank = __builtin_popcount(kept & wlow[j]);
      const uint32_t wi = (m.wo & 0xFFFFFFu) + KS * rank + wtp[j];
      const uint32_t o = a.off_w + static_cast<uint32_t>(sizeof(TA)) * wi + adj(j);
      off[j] = (kept & wbit[j]) != 0 ? o : 0x80000000u;
    }
  };
  auto no_adj = [](int) { return 0u; };
  // global -> registers: the next channel's halo tile (xf walks the channels
  // in order) and weights
  const TA* xf = x + static_cast<size_t>(c0) * sh * sw;
  const size_t hw = static_cast<size_t>(sh) * sw;
  auto fetch = [&](const uint32_t (&woff)[NWL]) __attribute__((always_inline)) {
    // the channel as the resource: soffset is not range checked, so the
    // channel offset goes into the base address
    const __amdgpu_buffer_rsrc_t cr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<TA*>(xf), static_cast<short>(0), static_cast<int>(chan_bytes), 0x00020000);
    xf += hw;
    if (v4) {
#pragma unroll
      for (int t = 0; t < NQ; ++t) {
        if constexpr (ABF) {
          const uint2 u = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(cr, qoff[t][0], 0, 0));
          xs[t][0] = bf16_lo(u.x); xs[t][1] = bf16_hi(u.x); xs[t][2] = bf16_lo(u.y); xs[t][3] = bf16_hi(u.y);
        } else {
          const float4 v = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(cr, qoff[t][0], 0, 0));
          xs[t][0] = v.x; xs[t][1] = v.y; xs[t][2] = v.z; xs[t][3] = v.w;
        }
      }
    } else {
#pragma unroll
      for (int t = 0; t < NQ; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if constexpr (ABF)
            xs[t][j] = __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(cr, qoff[t][j], 0, 0)) << 16);
          else
            xs[t][j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(cr, qoff[t][j], 0, 0));
        }
    }
#pragma unroll
    for (int j = 0; j < NWL; ++j) {
      if constexpr (ABF)
        ws[j] = __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(br, woff[j], 0, 0)) << 16);
      else
        ws[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(br, woff[j], 0, 0));
    }
  };
  // registers -> LDS ring slot
  auto store = [&](float* slot) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < NQ; ++t)
      *reinterpret_cast<float4*>(slot + 4 * (64 * t + lane)) = make_float4(xs[t][0], xs[t][1], xs[t][2], xs[t][3]);
#pragma unroll
    for (int j = 0; j < NWL; ++j) slot[G::PATCH + 64 * j + lane] = ws[j];
  };

  float acc[8][R][CC];
#pragma unroll
  for (int s = 0; s < 8; ++s)
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int q = 0; q < CC; ++q) acc[s][r][q] = 0.0f;
  // the FMAs of channel c for its kept slots, slot by slot (compile-time
  // slot index, so the accumulators stay in registers whatever the unroller
  // decides); canonical library: slot s's pattern code is byte s % 4 of code
  // word cx (slots 0-3) or cy (4-7), branched on bit by bit in place
  auto compute = [&](const Meta& m, uint32_t kc, const float (&pt)[PR][PC], const float (&wt)[8][KW])
      __attribute__((always_inline)) {
    static_for<0, 8>([&](auto si) __attribute__((always_inline)) {
      constexpr int s = decltype(si)::value;
      if (!((kc >> s) & 1u)) return;
      if constexpr (LIB == kLibDense9) {
        fma_tap<0, S, D>(acc[s], pt, wt[s][0]);
        fma_tap<1, S, D>(acc[s], pt, wt[s][1]);
        fma_tap<2, S, D>(acc[s], pt, wt[s][2]);
        fma_tap<3, S, D>(acc[s], pt, wt[s][3]);
        fma_tap<4, S, D>(acc[s], pt, wt[s][4]);
        fma_tap<5, S, D>(acc[s], pt, wt[s][5]);
        fma_tap<6, S, D>(acc[s], pt, wt[s][6]);
        fma_tap<7, S, D>(acc[s], pt, wt[s][7]);
        fma_tap<8, S, D>(acc[s], pt, wt[s][8]);
      } else {
        apply_canon8_bits<8 * (s & 3), S, D>(s < 4 ? m.cx : m.cy, acc[s], pt, wt[s][0], wt[s][1], wt[s][2],
                                             wt[s][3]);
      }
    });
  };

  if (ABF && c0 < c1) {
    Meta m0 = load_meta(c0), m1 = load_meta(c0 + 1), m2 = load_meta(c0 + 2);
    uint32_t wof[NWL];
    weight_offs(m0, wof, no_adj);
    fetch(wof);
    store(ring);
    if (c0 + 1 < c1) {
      weight_offs(m1, wof, no_adj);
      fetch(wof);
    }
#pragma unroll 1
    for (int c = c0; c < c1; ++c) {
      const int k = c - c0;
      float* cur = ring + (k & 1) * SLOT;
      float* nxt = ring + ((k + 1) & 1) * SLOT;
      weight_offs(m2, wof, no_adj);               // needs meta(c+2): before any LDS op is in flight
      if (c + 1 < c1) store(nxt);                 // channel c+1 -> LDS
      if (c + 2 < c1) fetch(wof);                 // channel c+2 -> registers
      // patch and the kept slots' weights of channel c
      const uint32_t kept = m0.wo >> 24;
      float p[PR][PC];
      float w[8][KW];
      if (kept != 0) {
        // weights first: the patch reads end with a wait that then covers both
        const float4* wc = reinterpret_cast<const float4*>(cur + G::PATCH);
#pragma unroll
        for (int s = 0; s < 8; ++s)
          if ((kept >> s) & 1u) {
#pragma unroll
            for (int i = 0; i < KW / 4; ++i) {
              const float4 v = wc[s * (KW / 4) + i];
              w[s][4 * i] = v.x; w[s][4 * i + 1] = v.y; w[s][4 * i + 2] = v.z; w[s][4 * i + 3] = v.w;
            }
          }
#pragma unroll
        for (int r = 0; r < PR; ++r) read_row<SH, SH, PC, VWL, true>(p[r], cur + lane_off + r * LSTR);
      }
      // everything of channel c is in registers once this wait returns; the
      // scalar loads issued next are then waited for only one channel later
      wait_lgkm();
      __builtin_amdgcn_sched_barrier(0);
      const Meta m3 = load_meta(c + 3);
      uint32_t kc = kept;
      asm volatile("" : "+s"(kc));   // fresh slot tests (no 64-bit condition masks kept live)
      if (kc != 0) {
        compute(m0, kc, p, w);
      }
      m0 = m1;
      m1 = m2;
      m2 = m3;
    }
  }

  if (!ABF && c0 < c1) {
    // the row-load width (16-byte or 4-byte DMAs) as a compile-time choice:
    // the channel loop is instantiated for both, so it carries no branch on it
    auto fp32_path = [&](auto v4c) __attribute__((always_inline)) {
      constexpr bool V4 = decltype(v4c)::value;
      // fp32: DMA pipeline.  Channel c lives in ring slot (c - c0) % NSLOT;
      // its halo tile and weights are DMA'd DPF channels before it is computed.
      // With PIPE its patch and weights are read from LDS into one of two
      // register sets one channel before it is computed, so those reads overlap
      // the previous channel's FMAs.  Per channel every lane issues QV (QS)
      // DMAs, so "channel c has landed" is vmcnt <= n * QV while n later
      // channels are in flight.
      constexpr int NS = G::NSLOT, DPF = G::DPF;
      constexpr int QV = G::NQ + NWL;       // 16-byte patch loads + weight loads
      constexpr int QS = 4 * G::NQ + NWL;   // 4-byte patch loads + weight loads
      const uint32_t ring_b = lds_addr(ring);
      // LDS byte offsets within a ring slot: 16-byte patch loads t at 1024 t,
      // 4-byte ones (t, j) at 256 (4 t + j), weight loads j at 4 PATCH + 256 j
      constexpr uint32_t LW0 = 4u * G::PATCH;
      const u32x4 brs = make_rsrc_below(blob, a.blob_bytes, kDmaShift);
      // descriptor of the next channel to DMA (channels are DMA'd in order)
      u32x4 cr = make_rsrc_below(x + static_cast<size_t>(c0) * sh * sw, chan_bytes, kDmaShift);
  #pragma unroll
      for (int t = 0; t < NQ; ++t)
  #pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t l = V4 ? 1024u * t : 256u * (4 * t + j);
          if (qoff[t][j] != 0x80000000u) qoff[t][j] += kDmaShift - (l & 4095u);
        }
      auto wadj = [](int j) { return kDmaShift - ((LW0 + 256u * j) & 4095u); };
      auto dma = [&](int c, uint32_t wo) __attribute__((always_inline)) {
        const uint32_t k = static_cast<uint32_t>(c - c0);
        const uint32_t sb = ring_b + 4u * ((k % NS) * SLOT);
        // the patch first: it does not depend on the channel's metadata, whose
        // scalar load may still be in flight (the first channels)
        Meta mw;
        mw.wo = wo;
        uint32_t wof[NWL];
        if constexpr (V4) {
          static_for<0, NQ>([&](auto ti) __attribute__((always_inline)) {
            constexpr int T = decltype(ti)::value;
            dma_b128_at<1024u * T, 1024u * (T - 1), T == 0>(cr, qoff[T][0], sb);
          });
          weight_offs(mw, wof, wadj);
          static_for<0, NWL>([&](auto ji) __attribute__((always_inline)) {
            constexpr int J = decltype(ji)::value;
            dma_b32_at<LW0 + 256u * J, (J == 0 ? 1024u * (NQ - 1) : LW0 + 256u * (J - 1)), false>(brs, wof[J], sb);
          });
        } else {
          static_for<0, 4 * NQ>([&](auto ii) __attribute__((always_inline)) {
            constexpr int I = decltype(ii)::value;
            dma_b32_at<256u * I, 256u * (I - 1), I == 0>(cr, qoff[I / 4][I % 4], sb);
          });
          weight_offs(mw, wof, wadj);
          static_for<0, NWL>([&](auto ji) __attribute__((always_inline)) {
            constexpr int J = decltype(ji)::value;
            dma_b32_at<LW0 + 256u * J, (J == 0 ? 256u * (4 * NQ - 1) : LW0 + 256u * (J - 1)), false>(brs, wof[J], sb);
          });
        }
        cr = next_channel(cr, chan_bytes);
      };
      auto load_wo = [&](int c) __attribute__((always_inline)) {
        const uint32_t e = min(e_base + static_cast<uint32_t>(c), e_last);
        return sload<uint32_t>(blob, a.off_woff + 4 * e);
      };
      // wait until channel c has landed in LDS; the DMAs of channels up to
      // min(c + n, c1 - 1) have been issued
      auto wait_landed = [&](int c, auto later) __attribute__((always_inline)) {
        constexpr int n = decltype(later)::value;
        asm volatile("" ::: "memory");
        if (c + n < c1) {
          if constexpr (V4)
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(n * QV));
          else
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(n * QS));
        } else {
          __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        }
        asm volatile("" ::: "memory");
      };
      // LDS -> registers: patch and weights of channel c (no wait).  Canonical
      // library: all 8 slots' weights unconditionally (pruned slots hold zeros;
      // fewer branches than testing each slot); all-ones library: kept slots.
      auto lds_read = [&](int c, uint32_t kept, float (&p)[PR][PC], float (&w)[8][KW]) __attribute__((always_inline)) {
        const uint32_t k = static_cast<uint32_t>(c - c0);
        const float* cur = ring + (k % NS) * SLOT;
        const float4* wc = reinterpret_cast<const float4*>(cur + G::PATCH);
  #pragma unroll
        for (int s = 0; s < 8; ++s)
          if (LIB == kLibCanon8 || ((kept >> s) & 1u)) {
  #pragma unroll
            for (int i = 0; i < KW / 4; ++i) {
              const float4 v = wc[s * (KW / 4) + i];
              w[s][4 * i] = v.x; w[s][4 * i + 1] = v.y; w[s][4 * i + 2] = v.z; w[s][4 * i + 3] = v.w;
            }
          }
  #pragma unroll
        for (int r = 0; r < PR; ++r) read_row<SH, SH, PC, VWL, false>(p[r], cur + lane_off + r * LSTR);
      };
      // running byte offsets of the scalar loads (clamped at the layer's last
      // channel, whose entries are then read again and not used)
      const uint32_t woff_last = a.off_woff + 4u * e_last, code_last = a.off_codes + 8u * e_last;
      uint32_t wo_n, wo_off, me_off, mc_off;
      Meta m0, m1;
      // prologue: channels c0 .. c0+DPF-1 in flight, channel c0 read into set A
      {
        uint32_t wo[DPF];
  #pragma unroll
        for (int i = 0; i < DPF; ++i) wo[i] = load_wo(c0 + i);
  #pragma unroll
        for (int i = 0; i < DPF; ++i)
          if (c0 + i < c1) dma(c0 + i, wo[i]);
        m0 = load_meta(c0);
        m1 = load_meta(c0 + 1);
        wo_n = load_wo(c0 + DPF);
        wo_off = min(a.off_woff + 4u * (e_base + c0 + DPF + 1), woff_last);
        me_off = min(a.off_woff + 4u * (e_base + c0 + 2), woff_last);
        mc_off = min(a.off_codes + 8u * (e_base + c0 + 2), code_last);
      }
      float pa[PR][PC], pb[PR][PC];
      float wa[8][KW], wb[8][KW];
      if constexpr (G::PIPE) {
        wait_lgkm();
        wait_landed(c0, std::integral_constant<int, DPF - 1>{});
        lds_read(c0, m0.wo >> 24, pa, wa);
      }
      // one channel.  Pipelined: X holds channel c (read one step earlier) and
      // Y receives channel c + 1.  Otherwise channel c is read into X here.
      auto step = [&](int c, float (&px)[PR][PC], float (&wx)[8][KW], float (&py)[PR][PC], float (&wy)[8][KW])
          __attribute__((always_inline)) {
        if constexpr (!G::PIPE) {
          wait_landed(c, std::integral_constant<int, DPF - 1>{});
          if ((m0.wo >> 24) != 0) lds_read(c, m0.wo >> 24, px, wx);
        }
        // channel c's patch and weights, and the previous step's scalar loads
        wait_lgkm();
  #pragma unroll
        for (int s = 0; s < 8; ++s)
  #pragma unroll
          for (int i = 0; i < KW; ++i) asm("" : "+v"(wx[s][i]));
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (G::PIPE) {
          if (c + 1 < c1) {
            wait_landed(c + 1, std::integral_constant<int, DPF - 2>{});
            lds_read(c + 1, m1.wo >> 24, py, wy);
          }
        }
        // channel c+DPF -> LDS (its slot was last read for channel c-1)
        if (c + DPF < c1) dma(c + DPF, wo_n);
        const uint32_t wo_nn = sload<uint32_t>(blob, wo_off);
        Meta m2;
        m2.wo = sload<uint32_t>(blob, me_off);
        {
          const uint2 cw = sload<uint2>(blob, mc_off);
          m2.cx = cw.x;
          m2.cy = cw.y;
        }
        wo_off = min(wo_off + 4u, woff_last);
        me_off = min(me_off + 4u, woff_last);
        mc_off = min(mc_off + 8u, code_last);
        __builtin_amdgcn_sched_barrier(0);
        uint32_t kc = m0.wo >> 24;
        asm volatile("" : "+s"(kc));   // fresh slot tests (no 64-bit condition masks kept live)
        if (kc != 0) {
          compute(m0, kc, px, wx);
        }
        m0 = m1;
        m1 = m2;
        wo_n = wo_nn;
      };
      if constexpr (G::PIPE) {
  #pragma unroll 1
        for (int c = c0; c < c1; c += 2) {
          step(c, pa, wa, pb, wb);
          if (c + 1 >= c1) break;
          step(c + 1, pb, wb, pa, wa);
        }
      } else {
  #pragma unroll 1
        for (int c = c0; c < c1; ++c) step(c, pa, wa, pa, wa);
      }
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));   // no DMA may land in the exchange area below
    };
    if (v4)
      fp32_path(std::true_type{});
    else
      fp32_path(std::false_type{});
  }

  // ---- combine the WS partial sums, PS slots at a time, in wave order; wave
  // k then finishes units u = k, k + WS, ... of the pass (unit = slot, row).
  // With a channel split over workgroups (ksplit > 1) the unit's sum goes to
  // this workgroup's block of the partial-sum buffer instead; a second kernel
  // adds the ksplit blocks of each tile in split order and finishes.
  // with PP_MAXPOOL2 the output is the 2 x 2 max pool (floor) of the
  // activated conv output: each lane's R x CC block holds whole windows
  const bool pool = (a.flags & PP_MAXPOOL2) != 0;
  const int pho = a.ho / 2, pwo = a.wo / 2;
  TA* __restrict__ y = static_cast<TA*>(a.y) + static_cast<size_t>(img) * a.c_out *
                                                   (pool ? static_cast<size_t>(pho) * pwo : static_cast<size_t>(a.ho) * a.wo);
  const bool relu = (a.flags & PP_RELU) != 0;
  // with PP_ACCUMULATE y holds a residual on entry: y = y + act(...), as a
  // separate add of the stored output would give (the activated value is
  // rounded to the storage type first)
  const bool accum = (a.flags & PP_ACCUMULATE) != 0;
  const bool shuf = (a.flags & PP_PIXSHUF2) != 0;
  const int oxl = ox0 + lx * CC;
  const bool vec = (CC % 4 == 0) && (a.wo % 4 == 0) && (reinterpret_cast<uintptr_t>(a.y) % (4 * sizeof(TA)) == 0);
  constexpr int NU = G::PS * R;   // units per pass
  constexpr int BLK = 8 * R * CC * 64;   // floats of one workgroup's partial-sum block
  const bool split = a.ksplit > 1;
  const uint32_t item = ((static_cast<uint32_t>(img) * a.tiles_y + ty) * a.tiles_x + tx) * a.n_groups + grp;
  // the group's 8 output channels (through perm) and biases, loaded together
  // once instead of one dependent pair per stored unit
  uint32_t permv[8];
  float biasv[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    permv[s] = sload<uint32_t>(blob, a.off_perm + 4 * (static_cast<uint32_t>(grp) * 8 + s));
    biasv[s] = sload<float>(blob, a.off_bias + 4 * (static_cast<uint32_t>(grp) * 8 + s));
  }
  static_assert(G::PS == 2, "the exchange passes cover two slots");
  // store of row r of the unit's slot: output channel o (>= c_out for a padding slot)
  auto finish = [&](uint32_t o, float bias, int r, float (&v)[CC]) __attribute__((always_inline)) {
    if (o >= static_cast<uint32_t>(a.c_out)) return;   // padding slot
    const int oy = oy0 + ly * R + r;
    if (oy >= a.ho) return;
#pragma unroll
    for (int q = 0; q < CC; ++q) {
      v[q] += bias;
      if (relu) v[q] = fmaxf(v[q], 0.0f);
      if constexpr (ABF) {
        if (accum) v[q] = bf16_lo(to_bf16_bits(v[q]));
      }
    }
    if (shuf) {
      // PixelShuffle(2): channel o lands in channel o / 4 of the 2ho x 2wo
      // output, row 2 oy + bit 1 of o, columns 2 ox + bit 0 of o
      TA* row2 = y + (static_cast<size_t>(o >> 2) * 2 * a.ho + 2 * oy + ((o >> 1) & 1)) * 2 * a.wo + (o & 1);
#pragma unroll
      for (int q = 0; q < CC; ++q) {
        if (oxl + q < a.wo) {
          if constexpr (ABF)
            reinterpret_cast<uint16_t*>(row2)[2 * (oxl + q)] = static_cast<uint16_t>(to_bf16_bits(v[q]));
          else
            reinterpret_cast<float*>(row2)[2 * (oxl + q)] = v[q];
        }
      }
      return;
    }
    TA* row = y + (static_cast<size_t>(o) * a.ho + oy) * a.wo;
    if (vec && oxl + CC <= a.wo) {
#pragma unroll
      for (int q = 0; q < CC; q += 4) {
        if (accum) {
          if constexpr (ABF) {
            const uint2 old = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(row) + oxl + q);
            v[q] = bf16_lo(old.x) + v[q];
            v[q + 1] = bf16_hi(old.x) + v[q + 1];
            v[q + 2] = bf16_lo(old.y) + v[q + 2];
            v[q + 3] = bf16_hi(old.y) + v[q + 3];
          } else {
            const float4 old = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(row) + oxl + q);
            v[q] = old.x + v[q];
            v[q + 1] = old.y + v[q + 1];
            v[q + 2] = old.z + v[q + 2];
            v[q + 3] = old.w + v[q + 3];
          }
        }
        if constexpr (ABF) {
          uint2 uu;
          uu.x = to_bf16_bits(v[q]) | (to_bf16_bits(v[q + 1]) << 16);
          uu.y = to_bf16_bits(v[q + 2]) | (to_bf16_bits(v[q + 3]) << 16);
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(row) + oxl + q) = uu;
        } else {
          *reinterpret_cast<float4*>(reinterpret_cast<float*>(row) + oxl + q) =
              make_float4(v[q], v[q + 1], v[q + 2], v[q + 3]);
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < CC; ++q) {
        if (oxl + q < a.wo) {
          if constexpr (ABF) {
            uint16_t* e = reinterpret_cast<uint16_t*>(row) + oxl + q;
            const float t = accum ? bf16_lo(*e) + v[q] : v[q];
            *e = static_cast<uint16_t>(to_bf16_bits(t));
          } else {
            float* e = reinterpret_cast<float*>(row) + oxl + q;
            *e = accum ? *e + v[q] : v[q];
          }
        }
      }
    }
  };
  // pooled store of rows r, r + 1 (r even) of slot s: max over each 2 x 2
  // window of the activated values, as a separate pool of the stored conv
  // output would take it
  auto finish_pool = [&](uint32_t o, float bias, int r, float (&v0)[CC], float (&v1)[CC])
      __attribute__((always_inline)) {
    if (o >= static_cast<uint32_t>(a.c_out)) return;   // padding slot
    const int oy = oy0 + ly * R + r;
    if (oy + 1 >= a.ho) return;   // incomplete window (floor)
    TA* row = y + (static_cast<size_t>(o) * pho + oy / 2) * pwo;
#pragma unroll
    for (int q = 0; q < CC; ++q) {
      v0[q] += bias;
      v1[q] += bias;
      if (relu) {
        v0[q] = fmaxf(v0[q], 0.0f);
        v1[q] = fmaxf(v1[q], 0.0f);
      }
    }
#pragma unroll
    for (int j = 0; j < CC / 2; ++j) {
      const int ox = oxl + 2 * j;
      if (ox + 1 < a.wo) {
        const float m = fmaxf(fmaxf(v0[2 * j], v0[2 * j + 1]), fmaxf(v1[2 * j], v1[2 * j + 1]));
        if constexpr (ABF)
          reinterpret_cast<uint16_t*>(row)[ox / 2] = static_cast<uint16_t>(to_bf16_bits(m));
        else
          reinterpret_cast<float*>(row)[ox / 2] = m;
      }
    }
  };
  // the unit's sum over the WS waves (exchange area) or this wave's accumulators
  auto gather = [&](int s, int ps, int r, float (&v)[CC]) __attribute__((always_inline)) {
    if (WS > 1) {
#pragma unroll
      for (int q = 0; q < CC; ++q) {
        float t = 0.0f;
        for (int k = 0; k < WS; ++k) t += lds[((k * G::PS * R + ps * R + r) * CC + q) * 64 + lane];
        v[q] = t;
      }
    } else {
#pragma unroll
      for (int q = 0; q < CC; ++q) v[q] = acc[s][r][q];
    }
  };
#pragma unroll
  for (int s0 = 0; s0 < 8; s0 += G::PS) {
    if (WS > 1) {
      __syncthreads();
      float* dst = lds + (wk * G::PS * R * CC) * 64 + lane;
#pragma unroll
      for (int ps = 0; ps < G::PS; ++ps)
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int q = 0; q < CC; ++q) dst[((ps * R + r) * CC + q) * 64] = acc[s0 + ps][r][q];
      __syncthreads();
    }
    if constexpr (R % 2 == 0 && CC % 2 == 0) {
      if (pool && !split) {
        // units (slot, row pair); a split pools in its second pass
        constexpr int NUP = G::PS * (R / 2);
#pragma unroll
        for (int u0 = 0; u0 < NUP; u0 += WS) {
          const int u = u0 + wk;
          if (u >= NUP) break;
          const int ps = u / (R / 2), r = 2 * (u % (R / 2));
          const int s = s0 + ps;
          float v0[CC], v1[CC];
          gather(s, ps, r, v0);
          gather(s, ps, r + 1, v1);
          finish_pool(ps == 0 ? permv[s0] : permv[s0 + 1], ps == 0 ? biasv[s0] : biasv[s0 + 1], r, v0, v1);
        }
        continue;
      }
    }
#pragma unroll
    for (int u0 = 0; u0 < NU; u0 += WS) {
      const int u = u0 + wk;
      if (u >= NU) break;
      const int ps = u / R, r = u % R;
      const int s = s0 + ps;
      float v[CC];
      gather(s, ps, r, v);
      if (split) {
        float* pb = a.part + static_cast<size_t>(item * a.ksplit + ks) * BLK + lane;
#pragma unroll
        for (int q = 0; q < CC; ++q) pb[((s * R + r) * CC + q) * 64] = v[q];
      } else {
        finish(ps == 0 ? permv[s0] : permv[s0 + 1], ps == 0 ? biasv[s0] : biasv[s0 + 1], r, v);
      }
    }
  }
}

// Second pass of a channel split: y = act(sum over the ksplit partial-sum
// blocks of a tile, in split order, + bias), stored through perm.  One
// workgroup per (image, tile, slot group); thread i handles element i of the
// tile's block layout ((slot, row, col) x lane).  With PP_MAXPOOL2 thread i
// handles pooled output i of the tile instead: the max over its 2 x 2
// window of the activated sums, in the order the conv kernel's own pooled
// store takes them.
template <int R, int CC, int LW, class TA>
__global__ __launch_bounds__(256) void pp_split_reduce_kernel(ConvParams a) {
  constexpr bool ABF = sizeof(TA) == 2;
  constexpr int LH = 64 / LW, TH = LH * R, TW = LW * CC;
  constexpr int BLK = 8 * R * CC * 64;
  const uint32_t item = blockIdx.x;
  const int grp = item % a.n_groups;
  uint32_t t = item / a.n_groups;
  const int tx = t % a.tiles_x;
  t /= a.tiles_x;
  const int ty = t % a.tiles_y;
  const int img = t / a.tiles_y;
  const float* pb = a.part + static_cast<size_t>(item) * a.ksplit * BLK;
  const bool relu = (a.flags & PP_RELU) != 0;
  if (a.flags & PP_MAXPOOL2) {
    const int pho = a.ho / 2, pwo = a.wo / 2;
    TA* __restrict__ yp = static_cast<TA*>(a.y) + static_cast<size_t>(img) * a.c_out * pho * pwo;
    constexpr int PH = TH / 2, PW = TW / 2;
    static_assert(TH % 2 == 0 && TW % 2 == 0, "pooled tiles need even sides");
    for (int i = threadIdx.x; i < 8 * PH * PW; i += 256) {
      const int s = i / (PH * PW), px = i % PW, py = (i / PW) % PH;
      const int oy = ty * TH + 2 * py, ox = tx * TW + 2 * px;
      if (oy + 1 >= a.ho || ox + 1 >= a.wo) continue;   // incomplete window (floor)
      const uint32_t slot = static_cast<uint32_t>(grp) * 8 + s;
      const uint32_t o = reinterpret_cast<const uint32_t*>(a.blob + a.off_perm)[slot];
      if (o >= static_cast<uint32_t>(a.c_out)) continue;   // padding slot
      const float bias = reinterpret_cast<const float*>(a.blob + a.off_bias)[slot];
      float v[2][2];
#pragma unroll
      for (int dy = 0; dy < 2; ++dy)
#pragma unroll
        for (int dx = 0; dx < 2; ++dx) {
          const int yl = 2 * py + dy, xl = 2 * px + dx;   // tile-local output
          const int lane = (yl / R) * LW + xl / CC;
          const int e = (s * R + yl % R) * CC + xl % CC;
          float t = 0.0f;
          for (int k = 0; k < a.ksplit; ++k) t += pb[static_cast<size_t>(k) * BLK + e * 64 + lane];
          t += bias;
          v[dy][dx] = relu ? fmaxf(t, 0.0f) : t;
        }
      const float m = fmaxf(fmaxf(v[0][0], v[0][1]), fmaxf(v[1][0], v[1][1]));
      const size_t at = (static_cast<size_t>(o) * pho + oy / 2) * pwo + ox / 2;
      if constexpr (ABF)
        reinterpret_cast<uint16_t*>(yp)[at] = static_cast<uint16_t>(to_bf16_bits(m));
      else
        reinterpret_cast<float*>(yp)[at] = m;
    }
    return;
  }
  TA* __restrict__ y = static_cast<TA*>(a.y) + static_cast<size_t>(img) * a.c_out * a.ho * a.wo;
  for (int i = threadIdx.x; i < BLK; i += 256) {
    const int lane = i % 64, e = i / 64;       // e = (s * R + r) * CC + q
    const int q = e % CC, r = (e / CC) % R, s = e / (CC * R);
    const int lx = lane % LW, ly = lane / LW;
    const int oy = ty * TH + ly * R + r, ox = tx * TW + lx * CC + q;
    if (oy >= a.ho || ox >= a.wo) continue;
    const uint32_t slot = static_cast<uint32_t>(grp) * 8 + s;
    const uint32_t o = reinterpret_cast<const uint32_t*>(a.blob + a.off_perm)[slot];
    if (o >= static_cast<uint32_t>(a.c_out)) continue;   // padding slot
    float v = 0.0f;
    for (int k = 0; k < a.ksplit; ++k) v += pb[static_cast<size_t>(k) * BLK + i];
    v += reinterpret_cast<const float*>(a.blob + a.off_bias)[slot];
    if (relu) v = fmaxf(v, 0.0f);
    const size_t at = (a.flags & PP_PIXSHUF2)
                        ? (static_cast<size_t>(o >> 2) * 2 * a.ho + 2 * oy + ((o >> 1) & 1)) * 2 * a.wo + 2 * ox + (o & 1)
                        : (static_cast<size_t>(o) * a.ho + oy) * a.wo + ox;
    if constexpr (ABF) {
      uint16_t* e = reinterpret_cast<uint16_t*>(y) + at;
      // PP_ACCUMULATE: y = y + act(...), the activated value rounded to bf16 first
      const float t = (a.flags & PP_ACCUMULATE) ? bf16_lo(*e) + bf16_lo(to_bf16_bits(v)) : v;
      *e = static_cast<uint16_t>(to_bf16_bits(t));
    } else {
      float* e = reinterpret_cast<float*>(y) + at;
      *e = (a.flags & PP_ACCUMULATE) ? *e + v : v;
    }
  }
}

#ifndef __HIPCC_RTC__   // host side
template <int LIB, int S, int D, int R, int CC, int LW, int WS, bool PIPE, class TA>
hipError_t launch_wave_tiling(ConvParams p, hipStream_t st) {
  using G = WGeo<LIB, S, D, R, CC, LW, WS, sizeof(TA) == 2, PIPE>;
  constexpr int SH = (4 - D % 4) % 4;   // the compiled padding is pad = D
  if constexpr (!G::fits) {
    return hipErrorInvalidConfiguration;
  } else {
    if (p.pad != D || G::TW % 4 != 0) return hipErrorInvalidConfiguration;
    p.tiles_x = (p.wo + G::TW - 1) / G::TW;
    p.tiles_y = (p.ho + G::TH - 1) / G::TH;
    p.n_ftiles = p.n_groups;
    if (p.ksplit < 1 || p.ksplit > p.c_in || (p.ksplit > 1 && !p.part)) return hipErrorInvalidValue;
    const size_t nb = static_cast<size_t>(p.n_groups) * p.tiles_x * p.tiles_y * p.n * p.ksplit;
    if (nb == 0 || nb > 0x7FFFFFFFull) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL((pp_conv3x3_wave_kernel<LIB, S, D, R, CC, LW, WS, SH, PIPE, TA>), dim3(static_cast<uint32_t>(nb)),
                       dim3(WS * 64), 0, st, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.ksplit == 1) return e;
    hipLaunchKernelGGL((pp_split_reduce_kernel<R, CC, LW, TA>), dim3(static_cast<uint32_t>(nb / p.ksplit)), dim3(256),
                       0, st, p);
    return hipGetLastError();
  }
}

#endif

}  // namespace kern
}  // namespace pp
