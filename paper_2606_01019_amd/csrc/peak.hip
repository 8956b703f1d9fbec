// Measured MFMA peak of the GPU the library runs on (gfx950): every SIMD of
// every CU runs waves that issue only f16 MFMA 32x32x16 on registers, eight
// independent accumulator chains per wave, no memory traffic in the timed
// loop.  Reports the achieved dense fp16 rate, to set beside the vendor's
// figure when MFMA fractions are quoted.
#include "common.h"
#include "kernels.h"

namespace hvd {

typedef float f32x16 __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256) void mfma_peak_kernel(int iters, float* sink) {
  f16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (_Float16)(1e-3f * (threadIdx.x + i));
    b[i] = (_Float16)(1e-3f * (blockIdx.x + i));
  }
  f32x16 acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[c][i] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < 8; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += acc[c][i];
  if (s == 1234.5f) sink[0] = s;  // keeps the work; never true for these inputs
}

}  // namespace hvd

using namespace hvd;

// flops of one launch: waves * iters * 8 chains * (32 * 32 * 16 * 2)
extern "C" int hvd_measure_mfma_peak(void* stream, double* tflops) {
  if (!tflops) return -1;
  hipStream_t s = (hipStream_t)stream;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                              hipSuccess)
    return -5;
  float* sink = nullptr;
  if (hipMalloc(&sink, sizeof(float)) != hipSuccess) return -3;
  const int blocks = cus * 8, iters = 4096;  // 8 four-wave workgroups per CU: 8 waves per SIMD
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = 0;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) rc = -5;
  double best = 0.0;
  for (int rep = 0; rc == 0 && rep < 4; ++rep) {  // the first launch warms up
    hipEventRecord(e0, s);
    hipLaunchKernelGGL(mfma_peak_kernel, dim3(blocks), dim3(256), 0, s, iters, sink);
    hipEventRecord(e1, s);
    if (hipEventSynchronize(e1) != hipSuccess) {
      rc = -5;
      break;
    }
    float ms = 0.f;
    hipEventElapsedTime(&ms, e0, e1);
    const double flops = (double)blocks * 4 * iters * 8 * (32.0 * 32 * 16 * 2);
    if (rep > 0 && ms > 0.f) best = std::max(best, flops / (ms * 1e-3) / 1e12);
  }
  if (e0) hipEventDestroy(e0);
  if (e1) hipEventDestroy(e1);
  hipFree(sink);
  *tflops = best;
  return rc;
}
