// dense.hip -- the dense layers and glue of the evaluated networks, for
// gfx950: dense k x k convolution (stride 1), 4x4 stride-2 transposed
// convolution, 2x2 max pooling, nearest x2 upsampling, PixelShuffle(2) and
// residual add.  None of these is pruned; they are the non-3x3 layers of the
// style-transfer, super-resolution and colourisation networks (Sec. 4).
//
// The dense convs and the transposed conv are dense contractions and run on
// the matrix cores (implicit GEMM, below), except dense convs with few
// filters or a short reduction (vector kernel); the glue ops are one
// elementwise kernel.
#include <hip/hip_runtime.h>

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
// Workgroup: 4 waves as WM x (4 / WM), each wave one 32 x 32 block of C, so a
// tile is BM = 32 WM filters by BN = 32 (4 / WM) pixels.  K advances in steps
// of kMK through two LDS buffers: the next step's global loads are in
// registers while the matrix cores run this one.  LDS is k-major ([k][m],
// [k][n]): the MFMA operand reads of a wave are lane-consecutive.  Weights
// are loaded k-fastest across lanes (whole 64-byte runs of a filter's row),
// stored through a row pitch of BM + 1 (no bank conflicts); pixels are loaded
// pixel-fastest (consecutive columns).
typedef float f32x16 __attribute__((ext_vector_type(16)));
constexpr int kMK = 32;

template <int MODE, int KD, int WM, class TA>
__global__ __launch_bounds__(256) void dense_mfma_kernel(DenseParams p, int n_tiles, int m_tiles) {
  constexpr int WN = 4 / WM, BM = 32 * WM, BN = 32 * WN;
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
  const TA* __restrict__ xi = static_cast<const TA*>(p.x) + static_cast<size_t>(bimg) * p.c_in * p.h * p.w;

  float ra[JA], rb[JB];
  auto fetch = [&](int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < JA; ++j) {
      const int kk = k0 + ak, ao = mt * BM + am0 + AR * j;
      float v = 0.0f;
      if (ao < p.c_out && kk < K) {
        if constexpr (MODE == 0) {
          v = ld(wt, static_cast<size_t>(ao) * K + kk);   // [c_out][c_in][k][k]
        } else {
          const int c = kk >> 2, a = (kk >> 1) & 1, b = kk & 1;
          const int ky = 1 - py + 2 * a, kx = 1 - px + 2 * b;
          v = ld(wt, ((static_cast<size_t>(c) * p.c_out + ao) * 4 + ky) * 4 + kx);   // [c_in][c_out][4][4]
        }
      }
      ra[j] = v;
    }
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      const int kk = k0 + bk0 + j;
      float v = 0.0f;
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
        if (iy >= 0 && iy < p.h && ix >= 0 && ix < p.w) v = ld(xi, (static_cast<size_t>(c) * p.h + iy) * p.w + ix);
      }
      rb[j] = v;
    }
  };
  auto put = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < JA; ++j) As[buf][ak][am0 + AR * j] = ra[j];
#pragma unroll
    for (int j = 0; j < JB; ++j) Bs[buf][bk0 + j][bn] = rb[j];
  };

  f32x16 acc = {};
  const int steps = (K + kMK - 1) / kMK;
  fetch(0);
  put(0);
  __syncthreads();
  for (int s = 0; s < steps; ++s) {
    const int buf = s & 1;
    if (s + 1 < steps) fetch((s + 1) * kMK);
#pragma unroll
    for (int k2 = 0; k2 < kMK; k2 += 2) {
      // operands of a 32 x 32 x 2 step: lane l holds A[l % 32][l / 32] and B[l / 32][l % 32]
      const float a = As[buf][k2 + (lane >> 5)][wm * 32 + (lane & 31)];
      const float b = Bs[buf][k2 + (lane >> 5)][wn * 32 + (lane & 31)];
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
    }
    if (s + 1 < steps) put(buf ^ 1);   // that buffer's last readers passed the barrier below one step ago
    __syncthreads();
  }

  // accumulator i of lane l is C[8 (i / 4) + 4 (l / 32) + i % 4][l % 32]
  const long gp = static_cast<long>(nt) * BN + wn * 32 + (lane & 31);
  if (gp >= np) return;
  const int ex = static_cast<int>(gp % gw);
  const long q = gp / gw;
  const int ey = static_cast<int>(q % gh);
  const long eimg = q / gh;
  const int oy = MODE == 0 ? ey : 2 * ey + py, ox = MODE == 0 ? ex : 2 * ex + px;
  TA* __restrict__ y = static_cast<TA*>(p.y) + static_cast<size_t>(eimg) * p.c_out * p.ho * p.wo;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int o = mt * BM + wm * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
    if (o < p.c_out) {
      float v = acc[i] + (p.bias ? p.bias[o] : 0.0f);
      if (p.relu) v = fmaxf(v, 0.0f);
      st(y, (static_cast<size_t>(o) * p.ho + oy) * p.wo + ox, v);
    }
  }
}

template <int MODE, int KD, class TA>
hipError_t launch_mfma(const DenseParams& p, hipStream_t st) {
  const int gh = MODE == 0 ? p.ho : p.h, gw = MODE == 0 ? p.wo : p.w;
  const long np = static_cast<long>(p.n) * gh * gw;
  const int classes = MODE == 0 ? 1 : 4;
  // few filters: 32 filters x 128 pixels per workgroup, else 64 x 64
  const bool narrow = p.c_out <= 32;
  const int bm = narrow ? 32 : 64, bn = narrow ? 128 : 64;
  const long n_tiles = (np + bn - 1) / bn, m_tiles = (p.c_out + bm - 1) / bm;
  const long blocks = n_tiles * m_tiles * classes;
  if (blocks < 1 || blocks > 0x7FFFFFFFL) return hipErrorInvalidConfiguration;
  const dim3 grid(static_cast<uint32_t>(blocks));
  if (narrow)
    hipLaunchKernelGGL((dense_mfma_kernel<MODE, KD, 1, TA>), grid, dim3(256), 0, st, p, static_cast<int>(n_tiles),
                       static_cast<int>(m_tiles));
  else
    hipLaunchKernelGGL((dense_mfma_kernel<MODE, KD, 2, TA>), grid, dim3(256), 0, st, p, static_cast<int>(n_tiles),
                       static_cast<int>(m_tiles));
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

template <int K, class TA>
hipError_t launch_conv_k(const DenseParams& p, hipStream_t st) {
  // the matrix cores once a tile has 16+ filters and the reduction is at
  // least 256 long (timed on the evaluated layers: the 9 x 9 convs 3 -> 32
  // and 32 -> 3 run faster on the vector ALUs, the 1 x 1 conv 256 -> 313
  // several times faster on the matrix cores)
  if (p.c_out >= 16 && static_cast<long>(p.c_in) * K * K >= 256) return launch_mfma<0, K, TA>(p, st);
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

hipError_t launch_deconv(const DenseParams& p, bool bf16, hipStream_t st) {
  if (p.k != 4 || p.stride != 2 || p.pad != 1 || p.ho != 2 * p.h || p.wo != 2 * p.w) return hipErrorInvalidValue;
  return bf16 ? launch_mfma<1, 2, uint16_t>(p, st) : launch_mfma<1, 2, float>(p, st);
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
