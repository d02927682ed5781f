// Matrix-core throughput probe: every SIMD runs two waves of independent
// v_mfma_f32_32x32x16_bf16 chains (8 accumulators per wave, operands in
// registers, no memory traffic in the loop), timed with HIP events.  It gives
// the dense bf16 rate this device sustains at its actual clock, the reference
// against which the kernels' matrix-core fractions can be read.
#include <hip/hip_runtime.h>

#include "../../include/terapipe.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256) void mfma_chain_kernel(int iters, float* sink) {
  const int lane = threadIdx.x & 63;
  bf16x8_t x, y;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    x[i] = (__bf16)(0.001f * (lane + i));
    y[i] = (__bf16)(0.002f * (lane - i));
  }
  f32x16_t acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, acc[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[j][v];
  // never true for these operands; keeps the chains live without a store
  if (s == 1.2345e30f) sink[blockIdx.x] = s;
}

}  // namespace

extern "C" tp_status tp_measure_mfma_peak(void* stream, int iters, void* sink,
                                          double* tflops) {
  if (!sink || !tflops || iters < 1) return TP_ERR_INVALID;
  hipStream_t s = (hipStream_t)stream;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return TP_ERR_HIP;
  const int grid = 2 * cus;  // 2 workgroups of 4 waves per CU: 2 waves per SIMD
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess) return TP_ERR_HIP;
  if (hipEventCreate(&e1) != hipSuccess) {
    hipEventDestroy(e0);
    return TP_ERR_HIP;
  }
  tp_status st = TP_OK;
  (void)hipGetLastError();  // drop an error an earlier, unrelated call left behind
  mfma_chain_kernel<<<grid, 256, 0, s>>>(iters, (float*)sink);  // warm-up
  bool ok = hipGetLastError() == hipSuccess && hipEventRecord(e0, s) == hipSuccess;
  if (ok) {
    mfma_chain_kernel<<<grid, 256, 0, s>>>(iters, (float*)sink);
    ok = hipGetLastError() == hipSuccess;
  }
  float ms = 0.f;
  ok = ok && hipEventRecord(e1, s) == hipSuccess && hipEventSynchronize(e1) == hipSuccess &&
       hipEventElapsedTime(&ms, e0, e1) == hipSuccess && ms > 0.f;
  if (!ok) {
    st = TP_ERR_HIP;
  } else {
    const double flops = (double)grid * 4 * iters * 8 * (2.0 * 32 * 32 * 16);
    *tflops = flops / (ms * 1e-3) / 1e12;
  }
  hipEventDestroy(e0);
  hipEventDestroy(e1);
  return st;
}
