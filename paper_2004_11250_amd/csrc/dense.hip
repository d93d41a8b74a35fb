// dense.hip -- the dense layers and glue of the evaluated networks, for
// gfx950: dense k x k convolution (stride 1), 4x4 stride-2 transposed
// convolution, 2x2 max pooling, nearest x2 upsampling, PixelShuffle(2) and
// residual add.  None of these is pruned; they are the non-3x3 layers of the
// style-transfer, super-resolution and colourisation networks (Sec. 4).
//
// The dense convs and the transposed conv are dense contractions and run on
// the matrix cores (implicit GEMM, below), except dense convs with few
// filters or a short reduction (vector kernels: a tiled one for 9 x 9 with
// pad 4 and a width that is a multiple of 4, a per-row one otherwise); the
// glue ops are one elementwise kernel.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "dense.hpp"

namespace pp {
namespace {

template <class T>
__device__ __forceinline__ T sload(const void* base, size_t byte_off) {
  typedef const __attribute__((address_space(4))) uint32_t* cptr;
  static_assert(sizeof(T) % 4 == 0, "scalar loads move whole dwords");
  const cptr src = (cptr)(static_cast<const uint8_t*>(base) + byte_off);
  union {
    T v;
    uint32_t u[sizeof(T) / 4];
  } r;
#pragma unroll
  for (int i = 0; i < static_cast<int>(sizeof(T) / 4); ++i) r.u[i] = src[i];
  return r.v;
}

__device__ __forceinline__ float ld(const float* p, size_t i) { return p[i]; }
__device__ __forceinline__ float ld(const uint16_t* p, size_t i) {
  return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
}
__device__ __forceinline__ void st(float* p, size_t i, float v) { p[i] = v; }
__device__ __forceinline__ void st(uint16_t* p, size_t i, float v) {
  uint32_t u = __float_as_uint(v);
  u += 0x7FFFu + ((u >> 16) & 1u);
  p[i] = static_cast<uint16_t>(u >> 16);
}

// weight w[idx] (fp32 or bf16 storage), wave-uniform index
template <class TA>
__device__ __forceinline__ float wload(const void* w, size_t idx) {
  if (sizeof(TA) == 4) return sload<float>(w, 4 * idx);
  const uint32_t u = sload<uint32_t>(w, (2 * idx) & ~static_cast<size_t>(3));
  return __uint_as_float((idx & 1) ? (u & 0xFFFF0000u) : (u << 16));
}

// Dense k x k, stride 1, zero padding `pad`, on the vector ALUs, for layers
// with few filters or a short reduction, where the GEMM tiles below would be
// mostly padding or gather: a wave computes filters [f0, f0+F) for output row
// oy, columns [ox0, ox0 + 64*CC) (the input row index is wave-uniform and
// out-of-image rows are skipped with a scalar branch); weights are
// wave-uniform scalar loads.
template <int K, int F, int CC, class TA>
__global__ __launch_bounds__(256) void dense_conv_vec_kernel(DenseParams p) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(blockIdx.x * 4 + (threadIdx.x >> 6)));
  const int col_tiles = (p.wo + 64 * CC - 1) / (64 * CC);
  const int f_tiles = (p.c_out + F - 1) / F;
  const long total = static_cast<long>(p.n) * p.ho * col_tiles * f_tiles;
  if (wave >= total) return;
  int t = wave;
  const int ft = t % f_tiles;
  t /= f_tiles;
  const int ct = t % col_tiles;
  t /= col_tiles;
  const int oy = t % p.ho;
  const int img = t / p.ho;
  const int f0 = ft * F;
  const int ox0 = ct * 64 * CC + lane * CC;

  const TA* x = static_cast<const TA*>(p.x) + static_cast<size_t>(img) * p.c_in * p.h * p.w;
  float acc[F][CC];
#pragma unroll
  for (int f = 0; f < F; ++f)
#pragma unroll
    for (int q = 0; q < CC; ++q) acc[f][q] = 0.0f;

  for (int c = 0; c < p.c_in; ++c) {
#pragma unroll 1
    for (int ky = 0; ky < K; ++ky) {
      const int iy = oy + ky - p.pad;
      if (iy < 0 || iy >= p.h) continue;   // wave-uniform
      float xs[CC + K - 1];
      const TA* row = x + (static_cast<size_t>(c) * p.h + iy) * p.w;
#pragma unroll
      for (int j = 0; j < CC + K - 1; ++j) {
        const int ix = ox0 - p.pad + j;
        xs[j] = (ix >= 0 && ix < p.w) ? ld(row, ix) : 0.0f;
      }
#pragma unroll
      for (int f = 0; f < F; ++f) {
        const int fo = min(f0 + f, p.c_out - 1);
        const size_t wbase = ((static_cast<size_t>(fo) * p.c_in + c) * K + ky) * K;
#pragma unroll
        for (int kx = 0; kx < K; ++kx) {
          const float wv = wload<TA>(p.wt, wbase + kx);
#pragma unroll
          for (int q = 0; q < CC; ++q) acc[f][q] = __builtin_fmaf(wv, xs[q + kx], acc[f][q]);
        }
      }
    }
  }
  TA* y = static_cast<TA*>(p.y) + static_cast<size_t>(img) * p.c_out * p.ho * p.wo;
#pragma unroll
  for (int f = 0; f < F; ++f) {
    const int fo = f0 + f;
    if (fo >= p.c_out) break;
    const float b = p.bias ? p.bias[fo] : 0.0f;
#pragma unroll
    for (int q = 0; q < CC; ++q) {
      const int ox = ox0 + q;
      if (ox < p.wo) {
        float v = acc[f][q] + b;
        if (p.relu) v = fmaxf(v, 0.0f);
        st(y, (static_cast<size_t>(fo) * p.ho + oy) * p.wo + ox, v);
      }
    }
  }
}

// Dense convolutions as implicit GEMMs on the fp32 matrix cores
// (v_mfma_f32_32x32x2_f32): C[o][pixel] = sum_k A[o][k] B[k][pixel], with A
// the weights and B the input gathered on the fly (the im2col matrix is
// never stored).  A k x k conv (stride 1) has k = (c, ky, kx) and pixels
// (image, oy, ox).  The 4 x 4, stride-2, pad-1 transposed conv splits into
// four classes of output pixels by parity (py, px); class (py, px) is a
// 2 x 2 conv over the input: output (2i + py, 2j + px) takes input rows
// i + py - a with kernel row 1 - py + 2a (a = 0, 1), and the same in x, so
// k = (c, a, b).  bf16 activations and weights are widened to fp32 on their
// way into LDS (exact products, fp32 accumulation, one rounding at the
// store).
//
// Workgroup: 4 waves as WM x (4 / WM), each wave TM x TN blocks of 32 x 32
// of C, so a tile is BM = 32 TM WM filters by BN = 32 TN (4 / WM) pixels
// (larger tiles load each operand element for more MACs).  K advances in steps
// of kMK through two LDS buffers: the next step's global loads are in
// registers while the matrix cores run this one.  LDS is k-major ([k][m],
// [k][n]): the MFMA operand reads of a wave are lane-consecutive.  Weights
// are loaded k-fastest across lanes (whole 64-byte runs of a filter's row),
// stored through a row pitch of BM + 1 (no bank conflicts); pixels are loaded
// pixel-fastest (consecutive columns).
typedef float f32x16 __attribute__((ext_vector_type(16)));
constexpr int kMK = 32;

// AP (fp32 transposed conv): the weights laid out per parity class as in the
// bf16 kernel, read as 16-byte pieces of 4 consecutive k.
template <int MODE, int KD, int WM, int TM, int TN, class TA, bool AP = false>
__global__ __launch_bounds__(256) void dense_mfma_kernel(DenseParams p, int n_tiles, int m_tiles) {
  static_assert(!AP || (MODE == 1 && sizeof(TA) == 4), "laid-out weights: fp32 transposed conv only");
  constexpr int WN = 4 / WM, BM = 32 * TM * WM, BN = 32 * TN * WN;
  constexpr int JA = kMK * BM / 256, JB = kMK * BN / 256;   // A / B elements per thread per step
  constexpr int AR = 256 / kMK;                             // A rows per load pass
  constexpr int KK = MODE == 0 ? KD * KD : 4;               // k per input channel
  __shared__ float As[2][kMK][BM + 1];
  __shared__ float Bs[2][kMK][BN];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wv % WM, wn = wv / WM;
  int t = blockIdx.x;
  const int nt = t % n_tiles;
  t /= n_tiles;
  const int mt = t % m_tiles;
  const int cls = t / m_tiles;   // parity class of the transposed conv (0 for a conv)
  const int py = cls >> 1, px = cls & 1;
  const int K = p.c_in * KK;
  const int gh = MODE == 0 ? p.ho : p.h, gw = MODE == 0 ? p.wo : p.w;   // the class's pixel grid
  const long np = static_cast<long>(p.n) * gh * gw;
  const TA* __restrict__ wt = static_cast<const TA*>(p.wt);

  // this thread's A column k (rows am0 + AR j) and B column (pixel), JB
  // consecutive k
  const int ak = tid % kMK, am0 = tid / kMK;
  const int bn = tid % BN, bk0 = (tid / BN) * JB;
  const long bp = static_cast<long>(nt) * BN + bn;
  const bool bvalid = bp < np;
  int by = 0, bx = 0;
  long bimg = 0;
  if (bvalid) {
    bx = static_cast<int>(bp % gw);
    const long q = bp / gw;
    by = static_cast<int>(q % gh);
    bimg = q / gh;
  }
  const TA* __restrict__ x = static_cast<const TA*>(p.x);
  // this thread's pixel's image, as an element offset into x
  const uint32_t ximg = static_cast<uint32_t>(bimg) * p.c_in * p.h * p.w;

  // loads through buffer resources (x and the weights, whole: the
  // descriptors stay wave-uniform): an element outside the layer or the
  // image gets an offset past the range and reads zero, so the loads need no
  // branches
  constexpr uint32_t kOut = 0x80000000u;
  const size_t x_elems = static_cast<size_t>(p.n) * p.c_in * p.h * p.w;
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<TA*>(x), static_cast<short>(0), static_cast<int>(x_elems * sizeof(TA)), 0x00020000);
  const size_t n_w = static_cast<size_t>(p.c_out) * p.c_in * (MODE == 0 ? KK : 16);   // the whole weight tensor
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<TA*>(wt), static_cast<short>(0), static_cast<int>(n_w * sizeof(TA)), 0x00020000);
  // load at byte offset off (bload_b) or element el (bload)
  auto bload_b = [&](__amdgpu_buffer_rsrc_t r, uint32_t off) __attribute__((always_inline)) {
    if constexpr (sizeof(TA) == 2)
      return __uint_as_float(static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0)) << 16);
    else
      return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
  };
  auto bload = [&](__amdgpu_buffer_rsrc_t r, uint32_t el) __attribute__((always_inline)) {
    return bload_b(r, el == kOut ? kOut : el * static_cast<uint32_t>(sizeof(TA)));
  };
  float ra[JA], rb[JB];
  // the general gather: every element's offset from (k, filter / pixel)
  auto fetch_any_a = [&](int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < JA; ++j) {
      const int kk = k0 + ak, ao = mt * BM + am0 + AR * j;
      uint32_t el = kOut;
      if (ao < p.c_out && kk < K) {
        if constexpr (MODE == 0) {
          el = static_cast<uint32_t>(ao) * K + kk;   // [c_out][c_in][k][k]
        } else {
          const int c = kk >> 2, a = (kk >> 1) & 1, b = kk & 1;
          const int ky = 1 - py + 2 * a, kx = 1 - px + 2 * b;
          el = ((static_cast<uint32_t>(c) * p.c_out + ao) * 4 + ky) * 4 + kx;   // [c_in][c_out][4][4]
        }
      }
      ra[j] = bload(wr, el);
    }
  };
  auto fetch_any_b = [&](int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      const int kk = k0 + bk0 + j;
      uint32_t el = kOut;
      if (bvalid && kk < K) {
        int c, iy, ix;
        if constexpr (MODE == 0) {
          c = kk / KK;
          const int r = kk - c * KK, ky = r / KD, kx = r - ky * KD;
          iy = by + ky - p.pad;
          ix = bx + kx - p.pad;
        } else {
          c = kk >> 2;
          iy = by + py - ((kk >> 1) & 1);
          ix = bx + px - (kk & 1);
        }
        if (iy >= 0 && iy < p.h && ix >= 0 && ix < p.w) el = ximg + (static_cast<uint32_t>(c) * p.h + iy) * p.w + ix;
      }
      rb[j] = bload(xr, el);
    }
  };
  // The transposed conv and the 1 x 1 conv: from one K step to the next a
  // thread's elements move by one fixed stride, the same for every lane (the
  // next kMK / 4 input channels, or the next kMK), so their offsets are taken
  // once and each full K step moves the descriptors' bases instead; a
  // partial last K step takes the general gather (past the last input
  // channel lies the next image, or the next filter's weights).
  constexpr bool STEPPED = MODE == 1 || KD == 1;
  constexpr uint32_t kES = static_cast<uint32_t>(sizeof(TA));
  uint32_t aoff[STEPPED ? JA : 1], boff[STEPPED ? JB : 1];
  if constexpr (STEPPED) {
#pragma unroll
    for (int j = 0; j < JA; ++j) {
      const int ao = mt * BM + am0 + AR * j;
      uint32_t el = kOut;
      if (ao < p.c_out) {
        if constexpr (MODE == 0) {
          el = static_cast<uint32_t>(ao) * K + ak;
        } else {
          const int c = ak >> 2, ky = 1 - py + 2 * ((ak >> 1) & 1), kx = 1 - px + 2 * (ak & 1);
          el = ((static_cast<uint32_t>(c) * p.c_out + ao) * 4 + ky) * 4 + kx;
        }
      }
      aoff[j] = el == kOut ? kOut : el * kES;
    }
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      const int kk = bk0 + j;
      uint32_t el = kOut;
      if (bvalid) {
        const int c = MODE == 0 ? kk : kk >> 2;
        const int iy = MODE == 0 ? by : by + py - ((kk >> 1) & 1);
        const int ix = MODE == 0 ? bx : bx + px - (kk & 1);
        if (iy >= 0 && iy < p.h && ix >= 0 && ix < p.w) el = ximg + (static_cast<uint32_t>(c) * p.h + iy) * p.w + ix;
      }
      boff[j] = el == kOut ? kOut : el * kES;
    }
  }
  // AP: pieces (row par + 32 j, k 4 paq .. 4 paq + 3) of the step (K = 4
  // c_in: a piece is wholly inside or past K)
  constexpr int APR = kMK / 4, JP = (BM * APR + 255) / 256;
  const int par = tid / APR, paq = tid % APR;
  uint32_t poff[AP ? JP : 1];
  float4 pa[AP ? JP : 1];
  const __amdgpu_buffer_rsrc_t pr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(p.scratch), static_cast<short>(0),
      AP ? static_cast<int>(static_cast<size_t>(16) * p.c_in * p.c_out * 4) : 0, 0x00020000);
  if constexpr (AP) {
#pragma unroll
    for (int j = 0; j < JP; ++j) {
      const int lr = par + (256 / APR) * j, ao = mt * BM + lr;
      poff[j] = lr < BM && ao < p.c_out ? ((static_cast<uint32_t>(cls) * p.c_out + ao) * K + 4 * paq) * 4u : kOut;
    }
  }
  const size_t a_step = MODE == 0 ? kMK : static_cast<size_t>(kMK / 4) * p.c_out * 16;      // elements per K step
  const size_t b_step = static_cast<size_t>(MODE == 0 ? kMK : kMK / 4) * p.h * p.w;
  auto fetch = [&](int s) __attribute__((always_inline)) {
    const int k0 = s * kMK;
    if constexpr (AP) {
#pragma unroll
      for (int j = 0; j < JP; ++j)
        pa[j] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(
                                               pr, poff[j] == kOut || k0 + 4 * paq >= K ? kOut : poff[j] + 4u * k0, 0, 0));
    }
    if constexpr (STEPPED) {
      if (k0 + kMK <= K) {
        const size_t ao0 = s * a_step, bo0 = s * b_step;
        const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<TA*>(wt + ao0), static_cast<short>(0), static_cast<int>((n_w - min(n_w, ao0)) * kES), 0x00020000);
        const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<TA*>(x + bo0), static_cast<short>(0), static_cast<int>((x_elems - min(x_elems, bo0)) * kES),
            0x00020000);
        if constexpr (!AP) {
#pragma unroll
          for (int j = 0; j < JA; ++j) ra[j] = bload_b(wrs, aoff[j]);
        }
#pragma unroll
        for (int j = 0; j < JB; ++j) rb[j] = bload_b(xrs, boff[j]);
        return;
      }
    }
    if constexpr (!AP) fetch_any_a(k0);
    fetch_any_b(k0);
  };
  auto put = [&](int buf) __attribute__((always_inline)) {
    if constexpr (AP) {
#pragma unroll
      for (int j = 0; j < JP; ++j) {
        const int lr = par + (256 / APR) * j;
        if (lr < BM) {
          As[buf][4 * paq][lr] = pa[j].x;
          As[buf][4 * paq + 1][lr] = pa[j].y;
          As[buf][4 * paq + 2][lr] = pa[j].z;
          As[buf][4 * paq + 3][lr] = pa[j].w;
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < JA; ++j) As[buf][ak][am0 + AR * j] = ra[j];
    }
#pragma unroll
    for (int j = 0; j < JB; ++j) Bs[buf][bk0 + j][bn] = rb[j];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};
  const int steps = (K + kMK - 1) / kMK;
  fetch(0);
  put(0);
  __syncthreads();
  for (int s = 0; s < steps; ++s) {
    const int buf = s & 1;
    if (s + 1 < steps) fetch(s + 1);
    // a 32 x 32 x 2 step takes A[l % 32][l / 32] and B[l / 32][l % 32] in
    // lane l; the operands of half a K step are read before its MFMAs (they
    // arrive in order, so each MFMA waits only for its own)
#pragma unroll
    for (int h = 0; h < kMK; h += kMK / 2) {
      float av[kMK / 4][TM], bv[kMK / 4][TN];
#pragma unroll
      for (int k2 = 0; k2 < kMK / 2; k2 += 2) {
#pragma unroll
        for (int i = 0; i < TM; ++i) av[k2 / 2][i] = As[buf][h + k2 + (lane >> 5)][(wm * TM + i) * 32 + (lane & 31)];
#pragma unroll
        for (int j = 0; j < TN; ++j) bv[k2 / 2][j] = Bs[buf][h + k2 + (lane >> 5)][(wn * TN + j) * 32 + (lane & 31)];
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int k2 = 0; k2 < kMK / 4; ++k2)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[k2][i], bv[k2][j], acc[i][j], 0, 0, 0);
    }
    if (s + 1 < steps) put(buf ^ 1);   // that buffer's last readers passed the barrier below one step ago
    __syncthreads();
  }

  // accumulator r of block (i, j), lane l, is C[8 (r / 4) + 4 (l / 32) + r % 4][l % 32] of the block
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const long gp = static_cast<long>(nt) * BN + (wn * TN + j) * 32 + (lane & 31);
    if (gp >= np) continue;
    const int ex = static_cast<int>(gp % gw);
    const long q = gp / gw;
    const int ey = static_cast<int>(q % gh);
    const long eimg = q / gh;
    const int oy = MODE == 0 ? ey : 2 * ey + py, ox = MODE == 0 ? ex : 2 * ex + px;
    TA* __restrict__ y = static_cast<TA*>(p.y) + static_cast<size_t>(eimg) * p.c_out * p.ho * p.wo;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int o = mt * BM + (wm * TM + i) * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (o < p.c_out) {
          float v = acc[i][j][r] + (p.bias ? p.bias[o] : 0.0f);
          if (p.relu) v = fmaxf(v, 0.0f);
          st(y, (static_cast<size_t>(o) * p.ho + oy) * p.wo + ox, v);
        }
      }
  }
}

// The same implicit GEMMs for bf16 activations and weights on the bf16
// matrix cores (v_mfma_f32_32x32x16_bf16, 16x the fp32 rate): operands stay
// bf16 through LDS, stored row-major per filter / pixel with k fastest
// ([row][k], a pitch of kMK + 8 elements: one 16-byte read gives a lane its
// 8 k of a 32 x 32 x 16 step), products are exact in fp32 and sums fp32, and
// the store rounds once to bf16.  The gathers are those of the fp32 kernel.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// AP (transposed conv): the weights come laid out per parity class,
// [class][filter][k] (deconv_relayout_kernel), so a thread loads 8
// consecutive k of a filter as one 16-byte piece; read as given (IOHW),
// consecutive k of a filter are 8 KB apart for 512 filters and a 64-lane load
// touches 16 cache lines for 128 useful bytes.
template <int MODE, int KD, int WM, int TM, int TN, bool AP = false>
__global__ __launch_bounds__(256) void dense_mfma_bf16_kernel(DenseParams p, int n_tiles, int m_tiles) {
  static_assert(!AP || MODE == 1, "laid-out weights: transposed conv only");
  constexpr int WN = 4 / WM, BM = 32 * TM * WM, BN = 32 * TN * WN;
  constexpr int JA = kMK * BM / 256, JB = kMK * BN / 256;   // A / B elements per thread per step
  constexpr int AR = 256 / kMK;                             // A rows per load pass
  constexpr int KK = MODE == 0 ? KD * KD : 4;               // k per input channel
  constexpr int kPitch = kMK + 8;
  static_assert(JB % 8 == 0, "a thread's B elements of a step are whole 16-byte pieces");
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM][kPitch];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN][kPitch];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wv % WM, wn = wv / WM;
  int t = blockIdx.x;
  const int nt = t % n_tiles;
  t /= n_tiles;
  const int mt = t % m_tiles;
  const int cls = t / m_tiles;   // parity class of the transposed conv (0 for a conv)
  const int py = cls >> 1, px = cls & 1;
  const int K = p.c_in * KK;
  const int gh = MODE == 0 ? p.ho : p.h, gw = MODE == 0 ? p.wo : p.w;
  const long np = static_cast<long>(p.n) * gh * gw;
  const uint16_t* __restrict__ wt = static_cast<const uint16_t*>(p.wt);
  const uint16_t* __restrict__ x = static_cast<const uint16_t*>(p.x);

  const int ak = tid % kMK, am0 = tid / kMK;
  const int bn = tid % BN, bk0 = (tid / BN) * JB;
  const long bp = static_cast<long>(nt) * BN + bn;
  const bool bvalid = bp < np;
  int by = 0, bx = 0;
  long bimg = 0;
  if (bvalid) {
    bx = static_cast<int>(bp % gw);
    const long q = bp / gw;
    by = static_cast<int>(q % gh);
    bimg = q / gh;
  }
  const uint32_t ximg = static_cast<uint32_t>(bimg) * p.c_in * p.h * p.w;
  constexpr uint32_t kOut = 0x80000000u;
  const size_t x_elems = static_cast<size_t>(p.n) * p.c_in * p.h * p.w;
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(x), static_cast<short>(0), static_cast<int>(x_elems * 2), 0x00020000);
  const size_t n_w = static_cast<size_t>(p.c_out) * p.c_in * (MODE == 0 ? KK : 16);
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(wt), static_cast<short>(0), static_cast<int>(n_w * 2), 0x00020000);
  auto bload_b = [&](__amdgpu_buffer_rsrc_t r, uint32_t off) __attribute__((always_inline)) {
    return static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0));
  };
  auto bload = [&](__amdgpu_buffer_rsrc_t r, uint32_t el) __attribute__((always_inline)) {
    return bload_b(r, el == kOut ? kOut : el * 2u);
  };
  uint32_t ra[JA], rb[JB];
  auto fetch_any_a = [&](int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < JA; ++j) {
      const int kk = k0 + ak, ao = mt * BM + am0 + AR * j;
      uint32_t el = kOut;
      if (ao < p.c_out && kk < K) {
        if constexpr (MODE == 0) {
          el = static_cast<uint32_t>(ao) * K + kk;
        } else {
          const int c = kk >> 2, a = (kk >> 1) & 1, b = kk & 1;
          const int ky = 1 - py + 2 * a, kx = 1 - px + 2 * b;
          el = ((static_cast<uint32_t>(c) * p.c_out + ao) * 4 + ky) * 4 + kx;
        }
      }
      ra[j] = bload(wr, el);
    }
  };
  auto fetch_any_b = [&](int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      const int kk = k0 + bk0 + j;
      uint32_t el = kOut;
      if (bvalid && kk < K) {
        int c, iy, ix;
        if constexpr (MODE == 0) {
          c = kk / KK;
          const int r = kk - c * KK, ky = r / KD, kx = r - ky * KD;
          iy = by + ky - p.pad;
          ix = bx + kx - p.pad;
        } else {
          c = kk >> 2;
          iy = by + py - ((kk >> 1) & 1);
          ix = bx + px - (kk & 1);
        }
        if (iy >= 0 && iy < p.h && ix >= 0 && ix < p.w) el = ximg + (static_cast<uint32_t>(c) * p.h + iy) * p.w + ix;
      }
      rb[j] = bload(xr, el);
    }
  };
  constexpr bool STEPPED = MODE == 1 || KD == 1;
  uint32_t aoff[STEPPED ? JA : 1], boff[STEPPED ? JB : 1];
  if constexpr (STEPPED) {
#pragma unroll
    for (int j = 0; j < JA; ++j) {
      const int ao = mt * BM + am0 + AR * j;
      uint32_t el = kOut;
      if (ao < p.c_out) {
        if constexpr (MODE == 0) {
          el = static_cast<uint32_t>(ao) * K + ak;
        } else {
          const int c = ak >> 2, ky = 1 - py + 2 * ((ak >> 1) & 1), kx = 1 - px + 2 * (ak & 1);
          el = ((static_cast<uint32_t>(c) * p.c_out + ao) * 4 + ky) * 4 + kx;
        }
      }
      aoff[j] = el == kOut ? kOut : el * 2u;
    }
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      const int kk = bk0 + j;
      uint32_t el = kOut;
      if (bvalid) {
        const int c = MODE == 0 ? kk : kk >> 2;
        const int iy = MODE == 0 ? by : by + py - ((kk >> 1) & 1);
        const int ix = MODE == 0 ? bx : bx + px - (kk & 1);
        if (iy >= 0 && iy < p.h && ix >= 0 && ix < p.w) el = ximg + (static_cast<uint32_t>(c) * p.h + iy) * p.w + ix;
      }
      boff[j] = el == kOut ? kOut : el * 2u;
    }
  }
  // AP: pieces (row ar + (256 / APR) j, k 8 aq .. 8 aq + 7) of the step; K is
  // a multiple of 8 (c_in even), so a piece is wholly inside or past K
  constexpr int APR = kMK / 8, JP = (BM * APR + 255) / 256;   // (a 32-row tile: half the threads)
  const int par = tid / APR, paq = tid % APR;
  uint32_t poff[AP ? JP : 1];
  uint4 pa[AP ? JP : 1];
  const __amdgpu_buffer_rsrc_t pr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(p.scratch), static_cast<short>(0),
      AP ? static_cast<int>(static_cast<size_t>(16) * p.c_in * p.c_out * 2) : 0, 0x00020000);
  if constexpr (AP) {
#pragma unroll
    for (int j = 0; j < JP; ++j) {
      const int lr = par + (256 / APR) * j, ao = mt * BM + lr;
      poff[j] = lr < BM && ao < p.c_out ? ((static_cast<uint32_t>(cls) * p.c_out + ao) * K + 8 * paq) * 2u : kOut;
    }
  }
  const size_t a_step = MODE == 0 ? kMK : static_cast<size_t>(kMK / 4) * p.c_out * 16;
  const size_t b_step = static_cast<size_t>(MODE == 0 ? kMK : kMK / 4) * p.h * p.w;
  auto fetch = [&](int s) __attribute__((always_inline)) {
    const int k0 = s * kMK;
    if constexpr (AP) {
#pragma unroll
      for (int j = 0; j < JP; ++j)
        pa[j] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                              pr, poff[j] == kOut || k0 + 8 * paq >= K ? kOut : poff[j] + 2u * k0, 0, 0));
    }
    if constexpr (STEPPED) {
      if (k0 + kMK <= K) {
        const size_t ao0 = s * a_step, bo0 = s * b_step;
        const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t*>(wt + ao0), static_cast<short>(0), static_cast<int>((n_w - min(n_w, ao0)) * 2),
            0x00020000);
        const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t*>(x + bo0), static_cast<short>(0), static_cast<int>((x_elems - min(x_elems, bo0)) * 2),
            0x00020000);
        if constexpr (!AP) {
#pragma unroll
          for (int j = 0; j < JA; ++j) ra[j] = bload_b(wrs, aoff[j]);
        }
#pragma unroll
        for (int j = 0; j < JB; ++j) rb[j] = bload_b(xrs, boff[j]);
        return;
      }
    }
    if constexpr (!AP) fetch_any_a(k0);
    fetch_any_b(k0);
  };
  auto put = [&](int buf) __attribute__((always_inline)) {
    if constexpr (AP) {
#pragma unroll
      for (int j = 0; j < JP; ++j)
        if (par + (256 / APR) * j < BM) *reinterpret_cast<uint4*>(&As[buf][par + (256 / APR) * j][8 * paq]) = pa[j];
    } else {
#pragma unroll
      for (int j = 0; j < JA; ++j) As[buf][am0 + AR * j][ak] = static_cast<uint16_t>(ra[j]);
    }
#pragma unroll
    for (int q = 0; q < JB / 8; ++q)
      *reinterpret_cast<uint4*>(&Bs[buf][bn][bk0 + 8 * q]) =
          make_uint4(rb[8 * q] | (rb[8 * q + 1] << 16), rb[8 * q + 2] | (rb[8 * q + 3] << 16),
                     rb[8 * q + 4] | (rb[8 * q + 5] << 16), rb[8 * q + 6] | (rb[8 * q + 7] << 16));
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};
  const int steps = (K + kMK - 1) / kMK;
  fetch(0);
  put(0);
  __syncthreads();
  for (int s = 0; s < steps; ++s) {
    const int buf = s & 1;
    if (s + 1 < steps) fetch(s + 1);
    // a 32 x 32 x 16 MFMA takes row l % 32 of A and column l % 32 of B, k
    // 8 (l / 32) .. 8 (l / 32) + 7 of its 16, in lane l
#pragma unroll
    for (int h = 0; h < kMK; h += 16) {
      bf16x8 av[TM], bv[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        av[i] = *reinterpret_cast<const bf16x8*>(&As[buf][(wm * TM + i) * 32 + (lane & 31)][h + 8 * (lane >> 5)]);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bv[j] = *reinterpret_cast<const bf16x8*>(&Bs[buf][(wn * TN + j) * 32 + (lane & 31)][h + 8 * (lane >> 5)]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    if (s + 1 < steps) put(buf ^ 1);   // that buffer's last readers passed the barrier below one step ago
    __syncthreads();
  }

  // accumulator r of block (i, j), lane l, is C[8 (r / 4) + 4 (l / 32) + r % 4][l % 32] of the block
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const long gp = static_cast<long>(nt) * BN + (wn * TN + j) * 32 + (lane & 31);
    if (gp >= np) continue;
    const int ex = static_cast<int>(gp % gw);
    const long q = gp / gw;
    const int ey = static_cast<int>(q % gh);
    const long eimg = q / gh;
    const int oy = MODE == 0 ? ey : 2 * ey + py, ox = MODE == 0 ? ex : 2 * ex + px;
    uint16_t* __restrict__ y = static_cast<uint16_t*>(p.y) + static_cast<size_t>(eimg) * p.c_out * p.ho * p.wo;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int o = mt * BM + (wm * TM + i) * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (o < p.c_out) {
          float v = acc[i][j][r] + (p.bias ? p.bias[o] : 0.0f);
          if (p.relu) v = fmaxf(v, 0.0f);
          st(y, (static_cast<size_t>(o) * p.ho + oy) * p.wo + ox, v);
        }
      }
  }
}

// The transposed conv's weights w[c][o][ky][kx] laid out for the GEMM of
// parity class (py, px): row (class, o) holds k = 4 c + 2 a + b, the tap
// (ky, kx) = (1 - py + 2 a, 1 - px + 2 b) -- the k order the kernel contracts
// in, so the sums are the same as when it reads w directly.
template <class T>
__global__ __launch_bounds__(256) void deconv_relayout_kernel(const T* __restrict__ w, T* __restrict__ out, int c_in,
                                                              int c_out) {
  const size_t n = static_cast<size_t>(16) * c_in * c_out;
  const int K = 4 * c_in;
  for (size_t i = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; i < n; i += static_cast<size_t>(gridDim.x) * 256) {
    const int k = static_cast<int>(i % K);
    const size_t r = i / K;
    const int o = static_cast<int>(r % c_out), cls = static_cast<int>(r / c_out);
    const int c = k >> 2, ky = 1 - (cls >> 1) + 2 * ((k >> 1) & 1), kx = 1 - (cls & 1) + 2 * (k & 1);
    out[i] = w[((static_cast<size_t>(c) * c_out + o) * 4 + ky) * 4 + kx];
  }
}

template <int MODE, int KD, class TA, bool AP = false>
hipError_t launch_mfma(const DenseParams& p, hipStream_t st) {
  const int gh = MODE == 0 ? p.ho : p.h, gw = MODE == 0 ? p.wo : p.w;
  const long np = static_cast<long>(p.n) * gh * gw;
  const int classes = MODE == 0 ? 1 : 4;
  // x and the weights are addressed with 32-bit byte offsets below 2^31 (the
  // offset 2^31 marks an element outside the layer)
  const size_t n_w = static_cast<size_t>(p.c_out) * p.c_in * (MODE == 0 ? KD * KD : 16);
  if (static_cast<size_t>(p.n) * p.c_in * p.h * p.w * sizeof(TA) >= (size_t{1} << 31) ||
      n_w * sizeof(TA) >= (size_t{1} << 31))
    return hipErrorInvalidValue;
  // tiles: 32 filters x 128 pixels (at most 32 filters), 128 x 128 (128+
  // filters, a reduction of 512+ and at least two such tiles per compute
  // unit), else 64 x 64 (timed on the colourization 4 x 4 transposed conv
  // 512 -> 256 and 1 x 1 conv 256 -> 313)
  const long big = (np + 127) / 128 * ((p.c_out + 127) / 128) * classes;
  const long k_len = static_cast<long>(p.c_in) * (MODE == 0 ? KD * KD : 4);
  const int shape = p.c_out <= 32 ? 0 : (p.c_out >= 128 && k_len >= 512 && big >= 512 ? 2 : 1);
  const int bm = shape == 0 ? 32 : (shape == 2 ? 128 : 64), bn = shape == 0 ? 128 : (shape == 2 ? 128 : 64);
  const long n_tiles = (np + bn - 1) / bn, m_tiles = (p.c_out + bm - 1) / bm;
  const long blocks = n_tiles * m_tiles * classes;
  if (blocks < 1 || blocks > 0x7FFFFFFFL) return hipErrorInvalidConfiguration;
  const dim3 grid(static_cast<uint32_t>(blocks));
  const int nt = static_cast<int>(n_tiles), mt = static_cast<int>(m_tiles);
  if constexpr (sizeof(TA) == 2) {
    if (shape == 0)
      hipLaunchKernelGGL((dense_mfma_bf16_kernel<MODE, KD, 1, 1, 1, AP>), grid, dim3(256), 0, st, p, nt, mt);
    else if (shape == 2)
      hipLaunchKernelGGL((dense_mfma_bf16_kernel<MODE, KD, 2, 2, 2, AP>), grid, dim3(256), 0, st, p, nt, mt);
    else
      hipLaunchKernelGGL((dense_mfma_bf16_kernel<MODE, KD, 2, 1, 1, AP>), grid, dim3(256), 0, st, p, nt, mt);
  } else {
    if (shape == 0)
      hipLaunchKernelGGL((dense_mfma_kernel<MODE, KD, 1, 1, 1, TA, AP>), grid, dim3(256), 0, st, p, nt, mt);
    else if (shape == 2)
      hipLaunchKernelGGL((dense_mfma_kernel<MODE, KD, 2, 2, 2, TA, AP>), grid, dim3(256), 0, st, p, nt, mt);
    else
      hipLaunchKernelGGL((dense_mfma_kernel<MODE, KD, 2, 1, 1, TA, AP>), grid, dim3(256), 0, st, p, nt, mt);
  }
  return hipGetLastError();
}

template <class TA>
__global__ __launch_bounds__(256) void glue_kernel(GlueParams p) {
  const size_t n_out = static_cast<size_t>(p.n) * p.c_out * p.ho * p.wo;
  const TA* x = static_cast<const TA*>(p.x);
  const TA* x2 = static_cast<const TA*>(p.x2);
  TA* y = static_cast<TA*>(p.y);
  for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n_out;
       i += static_cast<size_t>(gridDim.x) * blockDim.x) {
    const int ox = static_cast<int>(i % p.wo);
    size_t t = i / p.wo;
    const int oy = static_cast<int>(t % p.ho);
    t /= p.ho;
    const int c = static_cast<int>(t % p.c_out);
    const size_t img = t / p.c_out;
    float v;
    switch (p.op) {
      case kGlueMaxPool2: {
        const size_t base = ((img * p.c_in + c) * p.h + 2 * oy) * p.w + 2 * ox;
        v = fmaxf(fmaxf(ld(x, base), ld(x, base + 1)), fmaxf(ld(x, base + p.w), ld(x, base + p.w + 1)));
        break;
      }
      case kGlueUp2:
        v = ld(x, ((img * p.c_in + c) * p.h + oy / 2) * p.w + ox / 2);
        break;
      case kGluePixShuf2: {
        const int ci = 4 * c + 2 * (oy & 1) + (ox & 1);
        v = ld(x, ((img * p.c_in + ci) * p.h + oy / 2) * p.w + ox / 2);
        break;
      }
      default:  // add
        v = ld(x, i) + ld(x2, i);
        break;
    }
    st(y, i, v);
  }
}

// Dense 9 x 9 convolution, stride 1, pad 4 (same size), width a multiple of
// 4, on the vector ALUs: the style network's 9 x 9 layers (3 -> 32, 32 -> 3),
// whose few filters or short reduction leave GEMM tiles mostly padding.
// A wave computes F filters x one output row x 64 CC columns (CC adjacent
// columns per lane); S waves of a workgroup share that tile and take
// consecutive channel ranges, summed through LDS at the end, so a layer with
// few output tiles still fills the chip.  The workgroup's weights are staged
// once in LDS as fp32, [c][ky][f][12] (9 taps padded to 12 floats): a
// wave-uniform address, so each tap row is three broadcast 16-byte reads.
// Per (channel, ky) step a lane reads its CC + 8 input columns as aligned
// 4-element pieces through a raw-buffer descriptor of that input row: a row
// outside the image gets a zero-length descriptor and a piece outside the
// row an out-of-range offset, both read as zero (the padding) with no
// branch; the next step's pieces load while this step's FMAs run.
template <int F, int CC, int NW, int S, class TA>
__global__ __launch_bounds__(64 * NW) void dense9_tile_kernel(DenseParams p, int col_tiles, int n_tiles) {
  static_assert(NW % S == 0 && CC % 4 == 0, "tile shape");
  constexpr int T = NW / S;            // output tiles per workgroup
  constexpr int NP = (CC + 8) / 4;     // 4-element pieces per input row segment
  constexpr int WR = 12;               // LDS floats per (channel, ky, filter)
  constexpr uint32_t ES = sizeof(TA);
  constexpr uint32_t kOut = 0x80000000u;
  extern __shared__ float lds[];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
  const int sp = wave % S, tl = wave / S;
  const int f0 = static_cast<int>(blockIdx.y) * F;

  // ---- weights of filters [f0, f0 + F), every channel, fp32: the group's
  // weights are one contiguous block of the OIHW tensor, read in batches of
  // 8 independent coalesced loads per thread (the 3 pad floats of a tap row
  // are never read; a filter past c_out is zero)
  {
    const int fl = min(F, p.c_out - f0);
    const int n_g = fl * p.c_in * 81;
    const TA* wg = static_cast<const TA*>(p.wt) + static_cast<size_t>(f0) * p.c_in * 81;
    for (int i0 = threadIdx.x; i0 < n_g; i0 += 8 * 64 * NW) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = i0 + u * 64 * NW;
        v[u] = e < n_g ? ld(wg, e) : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int e = i0 + u * 64 * NW;
        if (e < n_g) {
          const int kx = e % 9, t9 = e / 9, ky = t9 % 9, t81 = t9 / 9, c = t81 % p.c_in, f = t81 / p.c_in;
          lds[((c * 9 + ky) * F + f) * WR + kx] = v[u];
        }
      }
    }
    for (int i = threadIdx.x; i < (F - fl) * p.c_in * 81; i += 64 * NW) {
      const int kx = i % 9, t9 = i / 9, ky = t9 % 9, t81 = t9 / 9, c = t81 % p.c_in, f = fl + t81 / p.c_in;
      lds[((c * 9 + ky) * F + f) * WR + kx] = 0.0f;
    }
  }
  __syncthreads();

  // ---- this wave's tile and channel range
  const int t = static_cast<int>(blockIdx.x) * T + tl;
  const bool live = t < n_tiles;
  const int ct = live ? t % col_tiles : 0;
  const int r = live ? t / col_tiles : 0;
  const int oy = r % p.ho, img = r / p.ho;
  const int cps = (p.c_in + S - 1) / S;
  const int c0 = min(sp * cps, p.c_in), c1 = min(c0 + cps, p.c_in);
  const int n_steps = live ? 9 * (c1 - c0) : 0;
  const int ox0 = ct * 64 * CC + lane * CC;
  uint32_t off[NP];
#pragma unroll
  for (int j = 0; j < NP; ++j) {
    const int ix = ox0 - 4 + 4 * j;
    off[j] = ix >= 0 && ix < p.w ? static_cast<uint32_t>(ix) * ES : kOut;
  }
  const TA* xi = static_cast<const TA*>(p.x) + static_cast<size_t>(img) * p.c_in * p.h * p.w;
  const int row_bytes = static_cast<int>(p.w * ES);

  auto load = [&](int c, int ky, float (&xs)[CC + 8]) __attribute__((always_inline)) {
    const int iy = oy + ky - 4;
    const bool rv = iy >= 0 && iy < p.h;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<TA*>(xi + (static_cast<size_t>(c) * p.h + (rv ? iy : 0)) * p.w), static_cast<short>(0),
        rv ? row_bytes : 0, 0x00020000);
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      if constexpr (ES == 2) {
        const uint2 u = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(xr, off[j], 0, 0));
        xs[4 * j + 0] = __uint_as_float(u.x << 16);
        xs[4 * j + 1] = __uint_as_float(u.x & 0xFFFF0000u);
        xs[4 * j + 2] = __uint_as_float(u.y << 16);
        xs[4 * j + 3] = __uint_as_float(u.y & 0xFFFF0000u);
      } else {
        const float4 u = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(xr, off[j], 0, 0));
        xs[4 * j + 0] = u.x;
        xs[4 * j + 1] = u.y;
        xs[4 * j + 2] = u.z;
        xs[4 * j + 3] = u.w;
      }
    }
  };

  float acc[F][CC];
#pragma unroll
  for (int f = 0; f < F; ++f)
#pragma unroll
    for (int q = 0; q < CC; ++q) acc[f][q] = 0.0f;

  auto fmas = [&](int c, int ky, const float (&xs)[CC + 8]) __attribute__((always_inline)) {
    const float* wr = lds + (c * 9 + ky) * F * WR;
#pragma unroll
    for (int f = 0; f < F; ++f) {
      const float4 wa = *reinterpret_cast<const float4*>(wr + f * WR);
      const float4 wb = *reinterpret_cast<const float4*>(wr + f * WR + 4);
      const float wc = wr[f * WR + 8];
      const float wk[9] = {wa.x, wa.y, wa.z, wa.w, wb.x, wb.y, wb.z, wb.w, wc};
#pragma unroll
      for (int kx = 0; kx < 9; ++kx)
#pragma unroll
        for (int q = 0; q < CC; ++q) acc[f][q] = __builtin_fmaf(wk[kx], xs[q + kx], acc[f][q]);
    }
  };

  // steps (c, ky) in order; the step after the last reloads the last one
  // (unconditional loads stay ahead of the FMAs)
  float xa[CC + 8], xb[CC + 8];
  int c = c0, ky = 0;
  if (n_steps > 0) load(c, ky, xa);
#pragma unroll 1
  for (int i = 0; i < n_steps; i += 2) {
    int cn = ky == 8 ? c + 1 : c, kn = ky == 8 ? 0 : ky + 1;
    if (i + 1 >= n_steps) cn = c, kn = ky;
    load(cn, kn, xb);
    fmas(c, ky, xa);
    if (i + 1 >= n_steps) break;
    c = cn, ky = kn;
    cn = ky == 8 ? c + 1 : c, kn = ky == 8 ? 0 : ky + 1;
    if (i + 2 >= n_steps) cn = c, kn = ky;
    load(cn, kn, xa);
    fmas(c, ky, xb);
    c = cn, ky = kn;
  }

  // ---- channel-split partial sums through LDS (the weights are done with)
  if constexpr (S > 1) {
    __syncthreads();
    if (sp != 0) {
#pragma unroll
      for (int f = 0; f < F; ++f)
#pragma unroll
        for (int q = 0; q < CC; ++q) lds[((wave * F + f) * CC + q) * 64 + lane] = acc[f][q];
    }
    __syncthreads();
    if (sp == 0) {
#pragma unroll 1
      for (int s2 = 1; s2 < S; ++s2)
#pragma unroll
        for (int f = 0; f < F; ++f)
#pragma unroll
          for (int q = 0; q < CC; ++q) acc[f][q] += lds[(((wave + s2) * F + f) * CC + q) * 64 + lane];
    }
  }
  if (!live || sp != 0) return;
  TA* y = static_cast<TA*>(p.y) + static_cast<size_t>(img) * p.c_out * p.ho * p.wo;
#pragma unroll
  for (int f = 0; f < F; ++f) {
    const int fo = f0 + f;
    if (fo >= p.c_out) break;
    const float b = p.bias ? p.bias[fo] : 0.0f;
#pragma unroll
    for (int j = 0; j < CC / 4; ++j) {
      const int ox = ox0 + 4 * j;
      if (ox >= p.wo) break;
      float v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[q] = acc[f][4 * j + q] + b;
        if (p.relu) v[q] = fmaxf(v[q], 0.0f);
      }
      const size_t at = (static_cast<size_t>(fo) * p.ho + oy) * p.wo + ox;
      if constexpr (ES == 2) {
        uint32_t u[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          u[q] = __float_as_uint(v[q]);
          u[q] = (u[q] + 0x7FFFu + ((u[q] >> 16) & 1u)) >> 16;
        }
        *reinterpret_cast<uint2*>(y + at) = make_uint2(u[0] | (u[1] << 16), u[2] | (u[3] << 16));
      } else {
        *reinterpret_cast<float4*>(y + at) = make_float4(v[0], v[1], v[2], v[3]);
      }
    }
  }
}

}  // namespace

template <int K, int F, class TA>
hipError_t launch_vec(const DenseParams& p, hipStream_t st) {
  constexpr int CC = K == 1 ? 1 : 4;
  const long waves = static_cast<long>(p.n) * p.ho * ((p.wo + 64 * CC - 1) / (64 * CC)) * ((p.c_out + F - 1) / F);
  const long blocks = (waves + 3) / 4;
  if (blocks < 1 || blocks > 0x7FFFFFFFL) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((dense_conv_vec_kernel<K, F, CC, TA>), dim3(static_cast<uint32_t>(blocks)), dim3(256), 0, st, p);
  return hipGetLastError();
}

template <int F, int CC, int NW, int S, class TA>
hipError_t launch_d9(const DenseParams& p, hipStream_t st) {
  constexpr int T = NW / S;
  const int col_tiles = (p.wo + 64 * CC - 1) / (64 * CC);
  const long tiles = static_cast<long>(p.n) * p.ho * col_tiles;
  const long bx = (tiles + T - 1) / T;
  const int fgs = (p.c_out + F - 1) / F;
  const size_t lw = static_cast<size_t>(p.c_in) * 9 * F * 12 * sizeof(float);
  const size_t red = S > 1 ? static_cast<size_t>(NW) * F * CC * 64 * sizeof(float) : 0;
  const size_t lds = lw > red ? lw : red;
  if (lds > 65536 || bx < 1 || tiles > 0x7FFFFFFFL || fgs > 65535) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((dense9_tile_kernel<F, CC, NW, S, TA>), dim3(static_cast<uint32_t>(bx), fgs), dim3(64 * NW),
                     lds, st, p, col_tiles, static_cast<int>(tiles));
  return hipGetLastError();
}

// F = 3 filters per wave for layers with at most 3 (the 32 -> 3 output
// layer), else 4; channels split S ways (1, 4 or 8: the smallest that puts
// 8192+ waves on the chip, at most c_in), S = 8 with two tiles per 16-wave
// workgroup (each staged weight set serves both), else 8-wave workgroups.
// Timed on the style network's layers at 512 x 512: 32 -> 3 at F 3, S 8 and
// 3 -> 32 at F 4, S 1 (F 8 and 8 columns per lane were slower).
template <int F>
int dense9_split(const DenseParams& p) {
  const long waves = static_cast<long>(p.n) * p.ho * ((p.wo + 255) / 256) * ((p.c_out + F - 1) / F);
  int s = 1;
  while (s < 8 && waves * s < 8192 && (s == 1 ? 4 : 8) <= p.c_in) s = s == 1 ? 4 : 8;
  return s;
}

template <int F, class TA>
hipError_t launch_dense9_f(const DenseParams& p, hipStream_t st) {
  const int s = dense9_split<F>(p);
  if (s == 8) return launch_d9<F, 4, 16, 8, TA>(p, st);
  if (s == 4) return launch_d9<F, 4, 8, 4, TA>(p, st);
  return launch_d9<F, 4, 8, 1, TA>(p, st);
}

template <class TA>
bool dense9_fits(const DenseParams& p) {
  const int f = p.c_out <= 3 ? 3 : 4;
  return p.k == 9 && p.pad == 4 && p.stride == 1 && p.w % 4 == 0 && p.ho == p.h && p.wo == p.w &&
         static_cast<size_t>(p.c_in) * 9 * f * 12 * sizeof(float) <= 65536;
}

template <int K, class TA>
hipError_t launch_conv_k(const DenseParams& p, hipStream_t st) {
  // the matrix cores once a tile has 16+ filters and the reduction is at
  // least 256 long (timed on the evaluated layers: the 9 x 9 convs 3 -> 32
  // and 32 -> 3 run faster on the vector ALUs, the 1 x 1 conv 256 -> 313
  // several times faster on the matrix cores); then the tiled 9 x 9 kernel
  // where its shape rules and LDS allow
  if (p.c_out >= 16 && static_cast<long>(p.c_in) * K * K >= 256) return launch_mfma<0, K, TA>(p, st);
  if (K == 9 && dense9_fits<TA>(p))
    return p.c_out <= 3 ? launch_dense9_f<3, TA>(p, st) : launch_dense9_f<4, TA>(p, st);
  return p.c_out <= 4 ? launch_vec<K, 4, TA>(p, st) : launch_vec<K, 8, TA>(p, st);
}

hipError_t launch_dense_conv(const DenseParams& p, bool bf16, hipStream_t st) {
  if (p.stride != 1) return hipErrorInvalidValue;
  switch (p.k) {
    case 1:
      return bf16 ? launch_conv_k<1, uint16_t>(p, st) : launch_conv_k<1, float>(p, st);
    case 3:
      return bf16 ? launch_conv_k<3, uint16_t>(p, st) : launch_conv_k<3, float>(p, st);
    case 9:
      return bf16 ? launch_conv_k<9, uint16_t>(p, st) : launch_conv_k<9, float>(p, st);
    default:
      return hipErrorInvalidValue;
  }
}

size_t deconv_scratch_bytes(int c_in, int c_out, bool bf16) {
  // (bf16: c_in even, so that k comes in whole 16-byte pieces of 8)
  if (bf16) return c_in % 2 == 0 ? static_cast<size_t>(16) * c_in * c_out * sizeof(uint16_t) : 0;
  return static_cast<size_t>(16) * c_in * c_out * sizeof(float);
}

// With scratch: the weights laid out per parity class first (timed on the
// colourization 512 -> 256 layer: the direct reads of the IOHW weights bound
// the bf16 form), then the GEMM reads them as 16-byte pieces.
template <class T>
hipError_t launch_deconv_t(const DenseParams& p, hipStream_t st) {
  const size_t nb = deconv_scratch_bytes(p.c_in, p.c_out, sizeof(T) == 2);
  if (p.scratch && nb && reinterpret_cast<uintptr_t>(p.scratch) % 16 == 0 && nb < (size_t{1} << 31)) {
    const size_t n = nb / sizeof(T);
    const uint32_t blocks = static_cast<uint32_t>(std::min<size_t>((n + 255) / 256, 4096));
    hipLaunchKernelGGL(deconv_relayout_kernel<T>, dim3(blocks), dim3(256), 0, st, static_cast<const T*>(p.wt),
                       static_cast<T*>(p.scratch), p.c_in, p.c_out);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_mfma<1, 2, T, true>(p, st);
  }
  return launch_mfma<1, 2, T>(p, st);
}

hipError_t launch_deconv(const DenseParams& p, bool bf16, hipStream_t st) {
  if (p.k != 4 || p.stride != 2 || p.pad != 1 || p.ho != 2 * p.h || p.wo != 2 * p.w) return hipErrorInvalidValue;
  return bf16 ? launch_deconv_t<uint16_t>(p, st) : launch_deconv_t<float>(p, st);
}

hipError_t launch_glue(const GlueParams& p, bool bf16, hipStream_t st) {
  const size_t n_out = static_cast<size_t>(p.n) * p.c_out * p.ho * p.wo;
  const size_t blocks = (n_out + 255) / 256;
  const dim3 grid(static_cast<uint32_t>(blocks < 65536 ? blocks : 65536));
  if (bf16) hipLaunchKernelGGL((glue_kernel<uint16_t>), grid, dim3(256), 0, st, p);
  else hipLaunchKernelGGL((glue_kernel<float>), grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace pp
