// dense.hip -- the dense layers and glue of the evaluated networks, for
// gfx950: dense k x k convolution (stride 1), 4x4 stride-2 transposed
// convolution, 2x2 max pooling, nearest x2 upsampling, PixelShuffle(2) and
// residual add.  None of these is pruned; they are the non-3x3 layers of the
// style-transfer, super-resolution and colourisation networks (Sec. 4).
//
// Dense convs: one wave computes F consecutive filters for 64*CC consecutive
// output pixels of one output row (so the input row index is wave-uniform and
// out-of-image rows are skipped with a scalar branch); weights are
// wave-uniform scalar loads.
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

// Dense k x k, stride 1, zero padding `pad`.  Wave: filters [f0, f0+F),
// output row oy, columns [ox0, ox0 + 64*CC).
template <int K, int F, int CC, class TA>
__global__ __launch_bounds__(256) void dense_conv_kernel(DenseParams p) {
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

// Transposed conv, kernel 4, stride 2, pad 1: output (oy, ox) takes input
// (iy, ix) with oy = 2*iy - 1 + ky, i.e. for each output row two kernel rows
// (the parity of oy + 1).  A lane owns the output column pair (2b, 2b+1):
//   out(2b)   = x[b] w[.,1] + x[b-1] w[.,3]
//   out(2b+1) = x[b+1] w[.,0] + x[b] w[.,2]
// Weights are [c_in][c_out][4][4].
template <int F, class TA>
__global__ __launch_bounds__(256) void deconv4s2_kernel(DenseParams p) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(blockIdx.x * 4 + (threadIdx.x >> 6)));
  const int col_tiles = (p.w + 63) / 64;   // input columns b
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
  const int b = ct * 64 + lane;

  const TA* x = static_cast<const TA*>(p.x) + static_cast<size_t>(img) * p.c_in * p.h * p.w;
  float acc[F][2];
#pragma unroll
  for (int f = 0; f < F; ++f) acc[f][0] = acc[f][1] = 0.0f;
  // kernel rows contributing to output row oy: ky = oy + 1 - 2*iy in [0,4)
  const int ky0 = (oy + 1) & 1;
  for (int c = 0; c < p.c_in; ++c) {
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int ky = ky0 + 2 * r;
      const int iy2 = oy + 1 - ky;   // = 2*iy
      const int iy = iy2 >> 1;
      if (iy2 < 0 || iy >= p.h) continue;   // wave-uniform
      const TA* row = x + (static_cast<size_t>(c) * p.h + iy) * p.w;
      const float xm = (b - 1 >= 0 && b - 1 < p.w) ? ld(row, b - 1) : 0.0f;
      const float x0 = (b < p.w) ? ld(row, b) : 0.0f;
      const float xp = (b + 1 < p.w) ? ld(row, b + 1) : 0.0f;
#pragma unroll
      for (int f = 0; f < F; ++f) {
        const int fo = min(f0 + f, p.c_out - 1);
        const size_t wb = ((static_cast<size_t>(c) * p.c_out + fo) * 4 + ky) * 4;
        const float w0 = wload<TA>(p.wt, wb), w1 = wload<TA>(p.wt, wb + 1);
        const float w2 = wload<TA>(p.wt, wb + 2), w3 = wload<TA>(p.wt, wb + 3);
        acc[f][0] = __builtin_fmaf(x0, w1, acc[f][0]);
        acc[f][0] = __builtin_fmaf(xm, w3, acc[f][0]);
        acc[f][1] = __builtin_fmaf(xp, w0, acc[f][1]);
        acc[f][1] = __builtin_fmaf(x0, w2, acc[f][1]);
      }
    }
  }
  TA* y = static_cast<TA*>(p.y) + static_cast<size_t>(img) * p.c_out * p.ho * p.wo;
#pragma unroll
  for (int f = 0; f < F; ++f) {
    const int fo = f0 + f;
    if (fo >= p.c_out) break;
    const float bb = p.bias ? p.bias[fo] : 0.0f;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int ox = 2 * b + q;
      if (ox < p.wo) {
        float v = acc[f][q] + bb;
        if (p.relu) v = fmaxf(v, 0.0f);
        st(y, (static_cast<size_t>(fo) * p.ho + oy) * p.wo + ox, v);
      }
    }
  }
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

hipError_t launch_dense_conv(const DenseParams& p, bool bf16, hipStream_t st) {
  constexpr int F = 8;
  if (p.k == 9) {
    constexpr int CC = 4;
    const long waves = static_cast<long>(p.n) * p.ho * ((p.wo + 64 * CC - 1) / (64 * CC)) * ((p.c_out + F - 1) / F);
    const dim3 grid(static_cast<uint32_t>((waves + 3) / 4));
    if (bf16) hipLaunchKernelGGL((dense_conv_kernel<9, F, CC, uint16_t>), grid, dim3(256), 0, st, p);
    else hipLaunchKernelGGL((dense_conv_kernel<9, F, CC, float>), grid, dim3(256), 0, st, p);
  } else if (p.k == 3) {
    constexpr int CC = 4;
    const long waves = static_cast<long>(p.n) * p.ho * ((p.wo + 64 * CC - 1) / (64 * CC)) * ((p.c_out + F - 1) / F);
    const dim3 grid(static_cast<uint32_t>((waves + 3) / 4));
    if (bf16) hipLaunchKernelGGL((dense_conv_kernel<3, F, CC, uint16_t>), grid, dim3(256), 0, st, p);
    else hipLaunchKernelGGL((dense_conv_kernel<3, F, CC, float>), grid, dim3(256), 0, st, p);
  } else if (p.k == 1) {
    constexpr int CC = 1;
    const long waves = static_cast<long>(p.n) * p.ho * ((p.wo + 64 * CC - 1) / (64 * CC)) * ((p.c_out + F - 1) / F);
    const dim3 grid(static_cast<uint32_t>((waves + 3) / 4));
    if (bf16) hipLaunchKernelGGL((dense_conv_kernel<1, F, CC, uint16_t>), grid, dim3(256), 0, st, p);
    else hipLaunchKernelGGL((dense_conv_kernel<1, F, CC, float>), grid, dim3(256), 0, st, p);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_deconv(const DenseParams& p, bool bf16, hipStream_t st) {
  constexpr int F = 8;
  if (p.k != 4 || p.stride != 2 || p.pad != 1) return hipErrorInvalidValue;
  const long waves = static_cast<long>(p.n) * p.ho * ((p.w + 63) / 64) * ((p.c_out + F - 1) / F);
  const dim3 grid(static_cast<uint32_t>((waves + 3) / 4));
  if (bf16) hipLaunchKernelGGL((deconv4s2_kernel<F, uint16_t>), grid, dim3(256), 0, st, p);
  else hipLaunchKernelGGL((deconv4s2_kernel<F, float>), grid, dim3(256), 0, st, p);
  return hipGetLastError();
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
