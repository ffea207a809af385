// Achievable peaks of the GPU the library runs on, measured with two plain
// kernels: dense bf16 MFMA throughput and HBM read bandwidth.  The rooflines
// of the decoding kernels are reported against the vendor peaks and against
// these measured ones.
#include <hip/hip_runtime.h>

#include "common.h"
#include "kernels.h"

namespace wd {

typedef float f32x16 __attribute__((ext_vector_type(16)));

// Each wave keeps 8 independent 32x32 accumulators busy on
// v_mfma_f32_32x32x16_bf16 (32768 flops each); the operands never change, so
// nothing but the matrix cores is exercised.  The result feeds a store that
// never happens (the sum cannot equal the sentinel) to keep the loop alive.
__global__ __launch_bounds__(256) void k_mfma_loop(float* out, int iters, float sentinel) {
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(1.0f + 0.001f * (float)(threadIdx.x + i));
    b[i] = (__bf16)(0.5f - 0.001f * (float)i);
  }
  f32x16 acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += acc[j][0] + acc[j][15];
  if (s == sentinel) out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// Reads n16 16-byte words once (non-temporal, as the weight streams do) and
// folds them into one word per thread.
__global__ __launch_bounds__(256) void k_read_stream(const u32x4* __restrict__ p, long n16,
                                                     unsigned* __restrict__ out) {
  const long stride = (long)gridDim.x * blockDim.x;
  unsigned x = 0;
  long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u32x4 v0 = __builtin_nontemporal_load(p + i);
    const u32x4 v1 = __builtin_nontemporal_load(p + i + stride);
    const u32x4 v2 = __builtin_nontemporal_load(p + i + 2 * stride);
    const u32x4 v3 = __builtin_nontemporal_load(p + i + 3 * stride);
    x ^= v0.x ^ v0.y ^ v0.z ^ v0.w ^ v1.x ^ v1.y ^ v1.z ^ v1.w;
    x ^= v2.x ^ v2.y ^ v2.z ^ v2.w ^ v3.x ^ v3.y ^ v3.z ^ v3.w;
  }
  for (; i < n16; i += stride) {
    const u32x4 v = __builtin_nontemporal_load(p + i);
    x ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  out[(long)blockIdx.x * blockDim.x + threadIdx.x] = x;
}

hipError_t measure_peaks(hipStream_t st, double* mfma_tflops, double* read_gbs) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  float* sink = nullptr;
  u32x4* buf = nullptr;
  unsigned* fold = nullptr;
  hipError_t err = hipSuccess;
  const int grid_mfma = 256 * 4, iters = 2048;
  const int grid_read = 256 * 16;
  const long bytes = 4L << 30;  // 4 GiB: far beyond every cache level
  float best_mfma = 1e30f, best_read = 1e30f;
#define WD_PK(x)                \
  do {                          \
    err = (x);                  \
    if (err != hipSuccess) goto done; \
  } while (0)
  WD_PK(hipEventCreate(&e0));
  WD_PK(hipEventCreate(&e1));
  WD_PK(hipMalloc(&sink, (size_t)grid_mfma * 256 * sizeof(float)));
  WD_PK(hipMalloc(&buf, bytes));
  WD_PK(hipMalloc(&fold, (size_t)grid_read * 256 * sizeof(unsigned)));
  WD_PK(hipMemsetAsync(buf, 0x3c, bytes, st));
  for (int rep = 0; rep < 3; ++rep) {
    float ms;
    WD_PK(hipEventRecord(e0, st));
    hipLaunchKernelGGL(k_mfma_loop, dim3(grid_mfma), dim3(256), 0, st, sink, iters, 1.2345f);
    WD_PK(hipGetLastError());
    WD_PK(hipEventRecord(e1, st));
    WD_PK(hipEventSynchronize(e1));
    WD_PK(hipEventElapsedTime(&ms, e0, e1));
    if (rep > 0 && ms < best_mfma) best_mfma = ms;
    WD_PK(hipEventRecord(e0, st));
    hipLaunchKernelGGL(k_read_stream, dim3(grid_read), dim3(256), 0, st, buf, bytes / 16, fold);
    WD_PK(hipGetLastError());
    WD_PK(hipEventRecord(e1, st));
    WD_PK(hipEventSynchronize(e1));
    WD_PK(hipEventElapsedTime(&ms, e0, e1));
    if (rep > 0 && ms < best_read) best_read = ms;
  }
  *mfma_tflops = (double)grid_mfma * 4 * iters * 8 * 32768.0 / (best_mfma * 1e-3) / 1e12;
  *read_gbs = (double)bytes / (best_read * 1e-3) / 1e9;
done:
#undef WD_PK
  if (e0) hipEventDestroy(e0);
  if (e1) hipEventDestroy(e1);
  if (sink) hipFree(sink);
  if (buf) hipFree(buf);
  if (fold) hipFree(fold);
  return err;
}

}  // namespace wd
