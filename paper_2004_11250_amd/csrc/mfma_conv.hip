// mfma_conv.hip -- a pruned 3x3 layer in bf16 on the bf16 matrix cores.
//
// Regrouping filters by pattern to feed the matrix cores (one dense
// contraction per (filter group, pattern) over the channels where some filter
// of the group uses the pattern) does not shrink the work when patterns are
// assigned independently per kernel: a channel lands in most groups' sets, so
// the contraction over all (tap, channel) pairs -- the layer's masked dense
// conv, A[o][(t, c)] = w[o][c][t] where tap t is in kernel (o, c)'s pattern
// and the kernel is kept, else 0 -- is the tightest matrix-core form.  It does
// 9 c_in c_out MACs per pixel instead of the surviving ones (about 4.5x more
// at half the kernels kept), on units with 16x the vector rate in bf16
// (2.5 PFLOP/s dense against 157 TFLOP/s), so it wins for large bf16 layers
// and loses for small ones, where its long reduction per tile leaves the chip
// idle; the planner picks per layer.
//
// Each call expands the blob into A in the caller's scratch
// (pp_mfma_expand_kernel: original filter order, k = (tap, channel), channel
// fastest, and the bias in original order) and runs an implicit GEMM
// C[o][pixel] = sum_k A[o][k] B[k][pixel], with B the input gathered on the
// fly (never stored).  k advances 32 or 64 at a time; with c_in a multiple
// of 32 the k of a step that one thread gathers for its pixel are one tap of
// consecutive channels, which differ only by the channel stride, taken as the
// loads' scalar offset.  Products of
// bf16 values are exact in fp32; sums are fp32; the epilogue (bias, ReLU,
// accumulate, PixelShuffle(2)) rounds once to bf16, as the vector kernels do.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "conv_pp.hpp"

namespace pp {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr uint32_t kOut = 0x80000000u;   // byte offset of an element outside a tensor (reads zero)

__device__ __forceinline__ uint32_t rne_bf16(float v) {
  uint32_t u = __float_as_uint(v);
  u += 0x7FFFu + ((u >> 16) & 1u);   // round to nearest even (finite values)
  return u >> 16;
}
__device__ __forceinline__ float bf16_val(uint32_t u) { return __uint_as_float(u << 16); }

// One thread per (slot group g, slot s, input channel c), channel fastest:
// the 9 taps of kernel (perm[8 g + s], c) into A[o][t][c] (zeros for taps off
// the pattern and for pruned kernels), and the slot's bias into bo[o].  Every
// (filter, channel) pair is written exactly once.  Offsets read from the
// device blob are clamped (a pattern id past the library reads as pruned, a
// weight index past n_wt as zero).
__global__ __launch_bounds__(256) void pp_mfma_expand_kernel(ConvParams a, uint16_t* __restrict__ am,
                                                             float* __restrict__ bo) {
  const long gid = static_cast<long>(blockIdx.x) * 256 + threadIdx.x;
  if (gid >= static_cast<long>(a.n_groups) * 8 * a.c_in) return;
  const int c = static_cast<int>(gid % a.c_in);
  const long gs = gid / a.c_in;   // 8 g + s
  const int s = static_cast<int>(gs & 7);
  const uint32_t o = reinterpret_cast<const uint32_t*>(a.blob + a.off_perm)[gs];
  if (o >= static_cast<uint32_t>(a.c_out)) return;   // padding slot
  const size_t gc = static_cast<size_t>(gs >> 3) * a.c_in + c;
  const uint8_t* code = a.blob + a.off_codes + gc * 8;
  const uint16_t* masks = reinterpret_cast<const uint16_t*>(a.blob + a.off_masks);
  const uint32_t wo = reinterpret_cast<const uint32_t*>(a.blob + a.off_woff)[gc];
  const uint32_t kept = wo >> 24;
  auto mask_of = [&](int q) -> uint32_t {
    const uint32_t id = code[q];
    return ((kept >> q) & 1u) && id < static_cast<uint32_t>(a.n_patterns) ? masks[id] & 0x1FFu : 0u;
  };
  // the slot's first weight: after the kept slots before it (bf16 kernels
  // are padded to an even element count)
  uint32_t idx = wo & 0xFFFFFFu;
  for (int q = 0; q < s; ++q) idx += (static_cast<uint32_t>(__builtin_popcount(mask_of(q))) + 1u) & ~1u;
  const uint32_t m = mask_of(s);
  const uint16_t* w = reinterpret_cast<const uint16_t*>(a.blob + a.off_w);
  uint16_t* dst = am + static_cast<size_t>(o) * 9 * a.c_in + c;
  for (int t = 0; t < 9; ++t) {
    uint16_t v = 0;
    if ((m >> t) & 1u) {
      v = idx < a.n_wt ? w[idx] : static_cast<uint16_t>(0);
      ++idx;
    }
    dst[static_cast<size_t>(t) * a.c_in] = v;
  }
  if (c == 0) bo[o] = reinterpret_cast<const float*>(a.blob + a.off_bias)[gs];
}

// Workgroup: 4 waves as 2 x 2, each wave TM x TN blocks of 32 x 32 of C: a
// tile is BM = 64 TM filters by BN = 64 TN pixels.  Two LDS buffers, row-major
// with k contiguous ([m][k], [n][k]), so each lane's MFMA operand (8
// consecutive k of one row) is one 16-byte read; the next step's global loads
// are in registers while the matrix cores run this one.  A: each thread loads
// 16-byte pieces of rows; B: each thread gathers KPT consecutive channels of
// one pixel (lanes take consecutive pixels, so each load is coalesced).  UP: the
// conv's input is the nearest x2 upsampling of x (PP_UPSAMPLE2).
template <int TM, int TN, int KM, bool UP, int G>
__global__ __launch_bounds__(256 * G) void pp_mfma_conv_kernel(ConvParams a, const uint16_t* __restrict__ am,
                                                               const float* __restrict__ bias, int n_tiles) {
  constexpr int BM = 64 * TM, BN = 64 * TN;
  constexpr int kMK = KM;               // k per step: KM / 16 MFMAs per block
  constexpr int kPitch = kMK + 8;       // LDS row pitch in bf16 (80 or 144 bytes: a lane's 16-byte reads spread over the banks)
  constexpr int KPT = kMK * BN / 256;   // B elements per thread per step
  constexpr int APR = kMK / 8;          // 16-byte A pieces per row and step
  constexpr int JA = BM * APR / 256;    // A pieces per thread
  static_assert(KPT % 8 == 0 && 32 % KPT == 0, "a thread's channels of a step are one tap (c_in a multiple of 32)");
  // per wave group: two buffers of A (BM rows) and B (BN rows); after the
  // loop the space holds the second group's accumulators
  constexpr int kRows = BM + BN;
  __shared__ __attribute__((aligned(16))) uint16_t smem[G * 2 * kRows * kPitch];
  static_assert(G == 1 || sizeof(smem) >= TM * TN * 16 * 256 * sizeof(float), "room for the group reduction");
  const int tid = threadIdx.x & 255, lane = tid & 63;
  const int grp = G == 1 ? 0 : __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 8));
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  auto As = [&](int buf, int row, int col) __attribute__((always_inline)) {
    return &smem[((grp * 2 + buf) * kRows + row) * kPitch + col];
  };
  auto Bs = [&](int buf, int row, int col) __attribute__((always_inline)) {
    return &smem[((grp * 2 + buf) * kRows + BM + row) * kPitch + col];
  };
  const int wm = wv & 1, wn = wv >> 1;
  const int nt = static_cast<int>(blockIdx.x % static_cast<uint32_t>(n_tiles));
  const int mt = static_cast<int>(blockIdx.x / static_cast<uint32_t>(n_tiles));
  const int K = 9 * a.c_in;
  const int steps = (K + kMK - 1) / kMK;   // K is a multiple of 32: the last step may be half
  const long np = static_cast<long>(a.n) * a.ho * a.wo;
  const int hs = UP ? a.h / 2 : a.h, wsd = UP ? a.w / 2 : a.w;   // stored input size
  const uint32_t hw = static_cast<uint32_t>(hs) * wsd;

  // A: rows ar + (256 / APR) j, k 8 aq .. 8 aq + 7 of the step
  const int ar = tid / APR, aq = tid % APR;
  const __amdgpu_buffer_rsrc_t arsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(am), static_cast<short>(0), a.c_out * K * 2, 0x00020000);
  uint32_t aoff[JA];
#pragma unroll
  for (int j = 0; j < JA; ++j) {
    const int row = mt * BM + ar + (256 / APR) * j;
    aoff[j] = row < a.c_out ? (static_cast<uint32_t>(row) * K + 8 * aq) * 2 : kOut;
  }
  // B: pixel bn, channels kb .. kb + KPT - 1 of the step (kb is wave-uniform)
  const int bn = tid % BN;
  const int kb = __builtin_amdgcn_readfirstlane(tid / BN) * KPT;
  const long bp = static_cast<long>(nt) * BN + bn;
  const bool bvalid = bp < np;
  int oy = 0, ox = 0;
  long img = 0;
  if (bvalid) {
    ox = static_cast<int>(bp % a.wo);
    const long q = bp / a.wo;
    oy = static_cast<int>(q % a.ho);
    img = q / a.ho;
  }
  const uint32_t ximg = static_cast<uint32_t>(img) * a.c_in * hw;
  const __amdgpu_buffer_rsrc_t xrsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.x), static_cast<short>(0), static_cast<int>(static_cast<uint32_t>(a.n) * a.c_in * hw * 2),
      0x00020000);

  uint32_t ra[JA][4], rb[KPT];
  auto fetch = [&](int st) __attribute__((always_inline)) {
    const int k0 = st * kMK;
    // a thread's KPT channels are one tap (c_in is a multiple of KPT); k
    // past K (the second half of a half step) reads zero
    const int t = (k0 + kb) / a.c_in, c0 = k0 + kb - t * a.c_in;
    const int ky = t / 3, kx = t - 3 * ky;
    const bool a_in = k0 + 8 * aq < K;
#pragma unroll
    for (int j = 0; j < JA; ++j) {
      const auto v =
          __builtin_amdgcn_raw_buffer_load_b128(arsrc, aoff[j] == kOut || !a_in ? kOut : aoff[j] + 2 * k0, 0, 0);
      ra[j][0] = v[0];
      ra[j][1] = v[1];
      ra[j][2] = v[2];
      ra[j][3] = v[3];
    }
    uint32_t bo = kOut;
    if (bvalid && k0 + kb < K) {
      const int iy = oy * a.stride + ky * a.dil - a.pad, ix = ox * a.stride + kx * a.dil - a.pad;
      if (iy >= 0 && iy < a.h && ix >= 0 && ix < a.w) {
        const int sy = UP ? iy >> 1 : iy, sx = UP ? ix >> 1 : ix;
        bo = (ximg + static_cast<uint32_t>(sy) * wsd + sx) * 2;
      }
    }
#pragma unroll
    for (int j = 0; j < KPT; ++j)
      rb[j] = __builtin_amdgcn_raw_buffer_load_b16(xrsrc, bo, static_cast<int>((c0 + j) * hw * 2), 0);
  };
  auto put = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < JA; ++j) {
      uint32_t* d = reinterpret_cast<uint32_t*>(As(buf, ar + (256 / APR) * j, 8 * aq));
      *reinterpret_cast<uint4*>(d) = make_uint4(ra[j][0], ra[j][1], ra[j][2], ra[j][3]);
    }
#pragma unroll
    for (int q = 0; q < KPT / 8; ++q) {
      uint32_t* d = reinterpret_cast<uint32_t*>(Bs(buf, bn, kb + 8 * q));
      *reinterpret_cast<uint4*>(d) =
          make_uint4((rb[8 * q] & 0xFFFFu) | (rb[8 * q + 1] << 16), (rb[8 * q + 2] & 0xFFFFu) | (rb[8 * q + 3] << 16),
                     (rb[8 * q + 4] & 0xFFFFu) | (rb[8 * q + 5] << 16), (rb[8 * q + 6] & 0xFFFFu) | (rb[8 * q + 7] << 16));
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};
  // wave group g takes k steps g, g + G, g + 2 G, ...: G tiles' worth of
  // loads in flight per workgroup; every thread runs every iteration (and
  // barrier), a group without a step that iteration only waits
  const int iters = (steps + G - 1) / G;
  if (grp < steps) {
    fetch(grp);
    put(0);
  }
  __syncthreads();
  for (int it = 0; it < iters; ++it) {
    const int buf = it & 1;
    const int s = it * G + grp;
    if (s + G < steps) fetch(s + G);
    if (s < steps) {
      // a 32 x 32 x 16 MFMA takes row l % 32 of A and column l % 32 of B, k
      // 8 (l / 32) .. 8 (l / 32) + 7 of its 16, in lane l
#pragma unroll
      for (int h = 0; h < kMK; h += 16) {
        bf16x8 av[TM], bv[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          av[i] = *reinterpret_cast<const bf16x8*>(As(buf, (wm * TM + i) * 32 + (lane & 31), h + 8 * (lane >> 5)));
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bv[j] = *reinterpret_cast<const bf16x8*>(Bs(buf, (wn * TN + j) * 32 + (lane & 31), h + 8 * (lane >> 5)));
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
      }
    }
    if (s + G < steps) put(buf ^ 1);   // that buffer's last readers passed the barrier below one iteration ago
    __syncthreads();
  }
  if constexpr (G == 2) {
    // group 1's sums into group 0's (one fixed order), through LDS (the
    // operand buffers are dead: every wave passed the last barrier)
    float* red = reinterpret_cast<float*>(smem);
    if (grp == 1) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) red[((i * TN + j) * 16 + r) * 256 + tid] = acc[i][j][r];
    }
    __syncthreads();
    if (grp == 1) return;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] += red[((i * TN + j) * 16 + r) * 256 + tid];
  }

  // accumulator r of block (i, j), lane l, is C[8 (r / 4) + 4 (l / 32) + r % 4][l % 32] of the block
  const bool relu = (a.flags & PP_RELU) != 0, accum = (a.flags & PP_ACCUMULATE) != 0;
  const bool shuf = (a.flags & PP_PIXSHUF2) != 0;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const long gp = static_cast<long>(nt) * BN + (wn * TN + j) * 32 + (lane & 31);
    if (gp >= np) continue;
    const int ex = static_cast<int>(gp % a.wo);
    const long q = gp / a.wo;
    const int ey = static_cast<int>(q % a.ho);
    const long eimg = q / a.ho;
    uint16_t* __restrict__ y = static_cast<uint16_t*>(a.y) + static_cast<size_t>(eimg) * a.c_out * a.ho * a.wo;
    if (shuf && !accum) {
      // PixelShuffle(2): filters o, o + 1 (o even; accumulators r, r + 1)
      // land in adjacent columns 2 ex, 2 ex + 1 of one output row: one
      // aligned 4-byte store per pair (c_out is a multiple of 4)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          const int o = mt * BM + (wm * TM + i) * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (o < a.c_out) {
            float v0 = acc[i][j][r] + bias[o], v1 = acc[i][j][r + 1] + bias[o + 1];
            if (relu) {
              v0 = fmaxf(v0, 0.0f);
              v1 = fmaxf(v1, 0.0f);
            }
            const size_t at = (static_cast<size_t>(o >> 2) * 2 * a.ho + 2 * ey + ((o >> 1) & 1)) * 2 * a.wo + 2 * ex;
            *reinterpret_cast<uint32_t*>(y + at) = rne_bf16(v0) | (rne_bf16(v1) << 16);
          }
        }
      continue;
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int o = mt * BM + (wm * TM + i) * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (o < a.c_out) {
          float v = acc[i][j][r] + bias[o];
          if (relu) v = fmaxf(v, 0.0f);
          const size_t at = shuf ? (static_cast<size_t>(o >> 2) * 2 * a.ho + 2 * ey + ((o >> 1) & 1)) * 2 * a.wo +
                                       2 * ex + (o & 1)
                                 : (static_cast<size_t>(o) * a.ho + ey) * a.wo + ex;
          // PP_ACCUMULATE: y = y + act(...), the activated value rounded to bf16 first
          const float t = accum ? bf16_val(y[at]) + bf16_val(rne_bf16(v)) : v;
          y[at] = static_cast<uint16_t>(rne_bf16(t));
        }
      }
  }
}

size_t a_bytes(const ConvParams& p) {
  return (static_cast<size_t>(p.c_out) * 9 * p.c_in * 2 + 255) / 256 * 256;
}

template <int TM, int TN, int KM, bool UP>
hipError_t launch_tiles(const ConvParams& p, const uint16_t* am, const float* bo, hipStream_t st) {
  constexpr int BM = 64 * TM, BN = 64 * TN;
  const long np = static_cast<long>(p.n) * p.ho * p.wo;
  const long n_tiles = (np + BN - 1) / BN, m_tiles = (p.c_out + BM - 1) / BM;
  const long blocks = n_tiles * m_tiles;
  if (blocks < 1 || blocks > 0x7FFFFFFFL) return hipErrorInvalidConfiguration;
  const dim3 grid(static_cast<uint32_t>(blocks));
  // grids of at most one tile per compute unit: two wave groups per tile
  // splitting its k steps (twice the loads in flight; with 512 tiles, whose
  // 8-wave workgroups no longer all fit at once, it timed slower)
  if (mfma_groups(p) == 2)
    hipLaunchKernelGGL((pp_mfma_conv_kernel<TM, TN, KM, UP, 2>), grid, dim3(512), 0, st, p, am, bo,
                       static_cast<int>(n_tiles));
  else
    hipLaunchKernelGGL((pp_mfma_conv_kernel<TM, TN, KM, UP, 1>), grid, dim3(256), 0, st, p, am, bo,
                       static_cast<int>(n_tiles));
  return hipGetLastError();
}

}  // namespace

bool mfma_eligible(const ConvParams& p) {
  if (p.c_in < 32 || p.c_in % 32 != 0 || p.c_out < 1) return false;   // (KPT = 32 channels)
  if (p.flags & PP_MAXPOOL2) return false;
  if (p.stride < 1 || p.stride > 2 || p.dil < 1 || p.dil > 2 || p.pad < 0) return false;
  const bool up = (p.flags & PP_UPSAMPLE2) != 0;
  if (up && (p.h % 2 || p.w % 2)) return false;
  // 32-bit byte offsets below 2^30 (2^31 marks an element outside a tensor
  // and the loads add the channel offset to it)
  const size_t hw = static_cast<size_t>(up ? p.h / 2 : p.h) * (up ? p.w / 2 : p.w);
  return static_cast<size_t>(p.n) * p.c_in * hw * 2 < (size_t{1} << 30) &&
         static_cast<size_t>(p.c_out) * 9 * p.c_in * 2 < (size_t{1} << 30);
}

bool mfma_long_k(const ConvParams& p) { return 9 * p.c_in >= 1152; }

int mfma_groups(const ConvParams& p) {
  const long bm = p.c_out > 64 ? 128 : 64;
  const long tiles = (static_cast<long>(p.n) * p.ho * p.wo + 127) / 128 * ((p.c_out + bm - 1) / bm);
  return tiles <= 256 ? 2 : 1;
}

size_t mfma_bytes(const ConvParams& p) { return a_bytes(p) + static_cast<size_t>(p.c_out) * sizeof(float); }

hipError_t launch_mfma_expand(const ConvParams& p, void* out, hipStream_t st) {
  if (!out || reinterpret_cast<uintptr_t>(out) % 256) return hipErrorInvalidValue;
  uint16_t* am = static_cast<uint16_t*>(out);
  float* bo = reinterpret_cast<float*>(static_cast<uint8_t*>(out) + a_bytes(p));
  const long ex = static_cast<long>(p.n_groups) * 8 * p.c_in;
  hipLaunchKernelGGL(pp_mfma_expand_kernel, dim3(static_cast<uint32_t>((ex + 255) / 256)), dim3(256), 0, st, p, am, bo);
  return hipGetLastError();
}

hipError_t launch_mfma_conv(const ConvParams& p, hipStream_t st) {
  if (!mfma_eligible(p) || !p.part || reinterpret_cast<uintptr_t>(p.part) % 256) return hipErrorInvalidValue;
  const uint16_t* am = reinterpret_cast<const uint16_t*>(p.part);
  const float* bo = reinterpret_cast<const float*>(reinterpret_cast<const uint8_t*>(p.part) + a_bytes(p));
  // PP_PREPARED: the workspace already holds the expansion (pp_conv2d_prepare)
  if (!(p.flags & PP_PREPARED)) {
    const hipError_t e = launch_mfma_expand(p, p.part, st);
    if (e != hipSuccess) return e;
  }
  const bool up = (p.flags & PP_UPSAMPLE2) != 0;
  // 128 x 128 tiles for more than 64 filters, else 64 x 128; k steps of 64
  // for reductions of 1152+ (fewer, longer steps: better where each tile's
  // long reduction is latency-bound), else 32 (half the LDS: more tiles per
  // compute unit) -- timed on the super-resolution, style-transfer and
  // colourization layers
  if (mfma_long_k(p)) {
    if (p.c_out > 64) return up ? launch_tiles<2, 2, 64, true>(p, am, bo, st) : launch_tiles<2, 2, 64, false>(p, am, bo, st);
    return up ? launch_tiles<1, 2, 64, true>(p, am, bo, st) : launch_tiles<1, 2, 64, false>(p, am, bo, st);
  }
  if (p.c_out > 64) return up ? launch_tiles<2, 2, 32, true>(p, am, bo, st) : launch_tiles<2, 2, 32, false>(p, am, bo, st);
  return up ? launch_tiles<1, 2, 32, true>(p, am, bo, st) : launch_tiles<1, 2, 32, false>(p, am, bo, st);
}

}  // namespace pp
