// ceiling.hip -- measured throughput ceilings of the GPU the benchmark runs
// on, reported next to the published peaks in the roofline figures:
//   * fp32 FMA issue rate: plain (non-packed) wave64 v_fmac_f32 in blocks of
//     the shape the pruned-conv kernels run (16 accumulators, 4 weights, a
//     6 x 6 register patch: one 4-tap pattern applied to a 4 x 4 output
//     block), four waves per SIMD;
//   * HBM bandwidth: a 16-byte-per-lane copy of a buffer far larger than the
//     caches (bytes read + bytes written per second).
// Built as its own library (libppceil.so): it allocates device memory and
// synchronises, which the conv library never does.
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace {

constexpr int kFmaIters = 2000;

__global__ __launch_bounds__(1024) void fma_kernel(const float* in, float* out, float w0, float w1, float w2,
                                                   float w3) {
  float p[6][6], acc[4][4];
  for (int i = 0; i < 36; ++i) p[i / 6][i % 6] = in[(threadIdx.x * 7 + i) & 1023];
  for (int i = 0; i < 16; ++i) acc[i / 4][i % 4] = 0.0f;
  for (int it = 0; it < kFmaIters; ++it) {
#pragma unroll
    for (int rep = 0; rep < 4; ++rep) {
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[r][q] = __builtin_fmaf(w0, p[r][q + 1], acc[r][q]);
          acc[r][q] = __builtin_fmaf(w1, p[r + 1][q], acc[r][q]);
          acc[r][q] = __builtin_fmaf(w2, p[r + 1][q + 1], acc[r][q]);
          acc[r][q] = __builtin_fmaf(w3, p[r + 1][q + 2], acc[r][q]);
        }
      asm volatile("" : "+v"(w0), "+v"(w1));   // keeps the 64 FMAs of each block
    }
  }
  float t = 0.0f;
  for (int i = 0; i < 16; ++i) t += acc[i / 4][i % 4];
  out[blockIdx.x * blockDim.x + threadIdx.x] = t;
}

__global__ void copy_kernel(const float4* __restrict__ a, float4* __restrict__ b, size_t n) {
  size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x;
  const size_t step = static_cast<size_t>(gridDim.x) * blockDim.x;
  for (; i < n; i += step) b[i] = a[i];
}

}  // namespace

// fp32 FMA throughput in TFLOP/s (2 flops per FMA) over `blocks` workgroups
// of 1024 threads (16 waves, 4 per SIMD when one workgroup runs per CU).
// Returns 0 on success, else the HIP error code.
extern "C" int pp_ceiling_fma(int blocks, double* tflops) {
  float *in = nullptr, *out = nullptr;
  hipError_t e = hipMalloc(&in, 4096 * sizeof(float));
  if (e == hipSuccess) e = hipMalloc(&out, static_cast<size_t>(blocks) * 1024 * sizeof(float));
  if (e == hipSuccess) e = hipMemset(in, 0, 4096 * sizeof(float));
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  float ms = 0.0f;
  if (e == hipSuccess) {
    hipLaunchKernelGGL(fma_kernel, dim3(blocks), dim3(1024), 0, 0, in, out, 1.0f, 2.0f, 3.0f, 4.0f);
    e = hipDeviceSynchronize();
  }
  if (e == hipSuccess) e = hipEventRecord(e0, 0);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(fma_kernel, dim3(blocks), dim3(1024), 0, 0, in, out, 1.0f, 2.0f, 3.0f, 4.0f);
    e = hipEventRecord(e1, 0);
  }
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (e == hipSuccess)
    *tflops = 2.0 * (4 * 64) * kFmaIters * (blocks * 1024.0) / (ms * 1e-3) / 1e12;   // 4 blocks of 64 FMAs per step
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (in) (void)hipFree(in);
  if (out) (void)hipFree(out);
  return static_cast<int>(e);
}

// copy bandwidth in GB/s (bytes read + bytes written) of a `bytes` buffer
extern "C" int pp_ceiling_copy(size_t bytes, int reps, double* gbs) {
  float4 *a = nullptr, *b = nullptr;
  const size_t n = bytes / sizeof(float4);
  hipError_t e = hipMalloc(&a, n * sizeof(float4));
  if (e == hipSuccess) e = hipMalloc(&b, n * sizeof(float4));
  if (e == hipSuccess) e = hipMemset(a, 0, n * sizeof(float4));
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  float ms = 0.0f;
  const int grid = 256 * 8;
  if (e == hipSuccess) {
    hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(256), 0, 0, a, b, n);
    e = hipDeviceSynchronize();
  }
  if (e == hipSuccess) e = hipEventRecord(e0, 0);
  for (int r = 0; r < reps && e == hipSuccess; ++r) hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(256), 0, 0, a, b, n);
  if (e == hipSuccess) e = hipEventRecord(e1, 0);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (e == hipSuccess) *gbs = 2.0 * n * sizeof(float4) * reps / (ms * 1e-3) / 1e9;
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (a) (void)hipFree(a);
  if (b) (void)hipFree(b);
  return static_cast<int>(e);
}
