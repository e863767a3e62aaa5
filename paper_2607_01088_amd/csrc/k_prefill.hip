// Row kernels of the prefix producer: the embedded prefix tokens of every job
// into the stacked fp32 residual stream, and each layer's K and V projections
// out of the stacked QKV rows into the jobs' caches.  Both are pure copies
// (HBM bound, 16-byte vectors); the backbone's arithmetic runs in the shared
// normalisation, GEMM and attention kernels.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "rosa_device.h"
#include "rosa_internal.h"

namespace rosa {

namespace {

// h[row][:] = float(emb_j[row - tok_off_j][:]), 4 elements per thread.
template <typename InT>
__global__ void __launch_bounds__(256) prefill_load_kernel(const PrefillJob *__restrict__ jobs,
                                                           const int32_t *__restrict__ row_job, int64_t M, int d,
                                                           float *__restrict__ h) {
  const int64_t per_row = d / 4;
  const int64_t total = M * per_row;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = i / per_row;
    const int c = (int)(i - row * per_row) * 4;
    const PrefillJob jb = jobs[row_job[row]];
    const InT *src = reinterpret_cast<const InT *>(jb.emb) + (row - jb.tok_off) * d + c;
    float4 v;
    if constexpr (sizeof(InT) == 4) {
      v = *reinterpret_cast<const float4 *>(src);
    } else {
      const uint2 raw = *reinterpret_cast<const uint2 *>(src);
      v.x = __uint_as_float(raw.x << 16);
      v.y = __uint_as_float(raw.x & 0xffff0000u);
      v.z = __uint_as_float(raw.y << 16);
      v.w = __uint_as_float(raw.y & 0xffff0000u);
    }
    *reinterpret_cast<float4 *>(h + row * d + c) = v;
  }
}

// cache_j[layer][row - tok_off_j][:] = the K (which 0) or V (which 1) columns of
// qkv row `row`; nkv*hd*esz bytes per row and tensor, moved in 16-byte chunks.
__global__ void __launch_bounds__(256) prefill_kv_scatter_kernel(const PrefillJob *__restrict__ jobs,
                                                                 const int32_t *__restrict__ row_job, int64_t M,
                                                                 const uint8_t *__restrict__ qkv, int64_t row_bytes,
                                                                 int64_t k_col_bytes, int64_t kv_bytes, int layer) {
  const int64_t chunks = kv_bytes / 16;
  const int64_t total = M * 2 * chunks;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = i / (2 * chunks);
    const int64_t r = i - row * 2 * chunks;
    const int which = r >= chunks;
    const int64_t c = (r - which * chunks) * 16;
    const PrefillJob jb = jobs[row_job[row]];
    const uint4 v = *reinterpret_cast<const uint4 *>(qkv + row * row_bytes + k_col_bytes + which * kv_bytes + c);
    uint8_t *dst = reinterpret_cast<uint8_t *>(which ? jb.v : jb.k) +
                   ((int64_t)layer * jb.P + (row - jb.tok_off)) * kv_bytes + c;
    *reinterpret_cast<uint4 *>(dst) = v;
  }
}

int grid_for(int64_t threads) {
  const int64_t blocks = (threads + 255) / 256;
  return (int)std::min<int64_t>(std::max<int64_t>(blocks, 1), 8192);
}

}  // namespace

hipError_t launch_prefill_load(const PrefillJob *jobs, const int32_t *row_job, int64_t M, int d, bool bf16_in,
                               float *h, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (d % 4) return hipErrorInvalidValue;
  const int grid = grid_for(M * (d / 4));
  if (bf16_in)
    hipLaunchKernelGGL(prefill_load_kernel<uint16_t>, dim3(grid), dim3(256), 0, s, jobs, row_job, M, d, h);
  else
    hipLaunchKernelGGL(prefill_load_kernel<float>, dim3(grid), dim3(256), 0, s, jobs, row_job, M, d, h);
  return hipGetLastError();
}

hipError_t launch_prefill_kv_scatter(const PrefillJob *jobs, const int32_t *row_job, int64_t M, const void *qkv,
                                     int ldqkv, int nq, int nkv, int hd, size_t esz, int layer, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  const int64_t kv_bytes = (int64_t)nkv * hd * (int64_t)esz;
  if (kv_bytes % 16 || ((int64_t)ldqkv * (int64_t)esz) % 16) return hipErrorInvalidValue;
  const int grid = grid_for(M * 2 * (kv_bytes / 16));
  hipLaunchKernelGGL(prefill_kv_scatter_kernel, dim3(grid), dim3(256), 0, s, jobs, row_job, M,
                     (const uint8_t *)qkv, (int64_t)ldqkv * (int64_t)esz, (int64_t)nq * hd * (int64_t)esz, kv_bytes,
                     layer);
  return hipGetLastError();
}

}  // namespace rosa
