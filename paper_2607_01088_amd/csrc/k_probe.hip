// Attainable-peak probe: a kernel that does nothing but back-to-back bf16
// MFMAs (v_mfma_f32_32x32x16_bf16, eight independent accumulators per wave,
// two waves per SIMD on every CU), timed with events.  Its rate is the dense
// bf16 matrix throughput the chip sustains at the clock it runs under that
// load, which the published peak (at the boost clock) does not show.
#include <hip/hip_runtime.h>

#include "rosa_device.h"
#include "../../include/rosa.h"
#include "../../include/rosa_debug.h"

namespace rosa {
namespace {

constexpr int kProbeAcc = 8;

__global__ void __launch_bounds__(256) mfma_probe_kernel(int iters, float *sink) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (bf16)(0.001f * (float)(lane + i));
    b[i] = (bf16)(0.002f * (float)(lane - i));
  }
  f32x16 acc[kProbeAcc];
#pragma unroll
  for (int j = 0; j < kProbeAcc; ++j) acc[j] = f32x16{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < kProbeAcc; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kProbeAcc; ++j) s += acc[j][0] + acc[j][15];
  // Never true for these inputs; keeps the products live.
  if (s == 1234.5f) sink[blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace
}  // namespace rosa

extern "C" rosa_status rosa_debug_mfma_peak(int32_t device, double *tflops) {
  using namespace rosa;
  if (!tflops) return ROSA_E_INVALID;
  *tflops = 0.0;
  int n_cu = 0;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  float *sink = nullptr;
  hipStream_t s = nullptr;
  hipError_t e = hipSetDevice(device);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, device);
  const int blocks = 2 * (n_cu > 0 ? n_cu : 1);       // 8 waves per CU: two per SIMD
  if (e == hipSuccess) e = hipMalloc(&sink, (size_t)blocks * 256 * sizeof(float));
  if (e == hipSuccess) e = hipStreamCreate(&s);
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  const int iters = 20000;
  if (e == hipSuccess) {
    hipLaunchKernelGGL(mfma_probe_kernel, dim3(blocks), dim3(256), 0, s, 100, sink);   // warm-up
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(e0, s);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(mfma_probe_kernel, dim3(blocks), dim3(256), 0, s, iters, sink);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(e1, s);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  if (e == hipSuccess && ms > 0.f) {
    const double flops = (double)blocks * 4 * iters * kProbeAcc * (2.0 * 32 * 32 * 16);
    *tflops = flops / (ms * 1e-3) / 1e12;
  }
  if (e0) hipEventDestroy(e0);
  if (e1) hipEventDestroy(e1);
  if (s) hipStreamDestroy(s);
  if (sink) hipFree(sink);
  return e == hipSuccess ? ROSA_OK : ROSA_E_DEVICE;
}
