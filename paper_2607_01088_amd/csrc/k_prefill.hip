// Row kernels of the prefix producer: the embedded prefix tokens of every job
// into the stacked fp32 residual stream, each layer's K and V projections out
// of the stacked QKV rows into the jobs' caches (both pure copies, HBM bound,
// 16-byte vectors), and the optional rotary position embedding of each
// layer's queries and keys.  The rest of the backbone's arithmetic runs in the
// shared normalisation, GEMM and attention kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

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

// Rotary position table: tab[p][i] = (cos, sin) of p * base^(-i / half) for
// positions p < n_pos and pairs i < half (half = head_dim / 2), computed in
// double and rounded once.
__global__ void __launch_bounds__(256) rope_table_kernel(float2 *__restrict__ tab, int n_pos, int half,
                                                         double log2_base) {
  const int64_t n = (int64_t)n_pos * half;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n; idx += (int64_t)gridDim.x * blockDim.x) {
    const int pos = (int)(idx / half), i = (int)(idx - (int64_t)pos * half);
    const double inv = exp2(-(double)i / (double)half * log2_base);
    double sn, cs;
    sincos((double)pos * inv, &sn, &cs);
    tab[idx] = make_float2((float)cs, (float)sn);
  }
}

// In place on the first nheads heads of every qkv row (the query heads, then
// the key heads): element pair (i, i + half) of a head at the row's position p
// (its index within its job) becomes (x1 c - x2 s, x2 c + x1 s) with
// (c, s) = tab[p][i].  Four pairs per thread.
template <typename T>
__global__ void __launch_bounds__(256) rope_apply_kernel(const PrefillJob *__restrict__ jobs,
                                                         const int32_t *__restrict__ row_job, int64_t M,
                                                         T *__restrict__ qkv, int64_t ldqkv, int nheads, int half,
                                                         const float2 *__restrict__ tab) {
  const int quads = half / 4;
  const int64_t per_row = (int64_t)nheads * quads;
  const int64_t total = M * per_row;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = idx / per_row;
    const int r = (int)(idx - row * per_row);
    const int head = r / quads, i = (r - head * quads) * 4;
    const int64_t pos = row - jobs[row_job[row]].tok_off;
    T *x = qkv + row * ldqkv + (int64_t)head * 2 * half + i;
    float a[4], b[4];
    if constexpr (sizeof(T) == 4) {
      const float4 va = *reinterpret_cast<const float4 *>(x), vb = *reinterpret_cast<const float4 *>(x + half);
      a[0] = va.x; a[1] = va.y; a[2] = va.z; a[3] = va.w;
      b[0] = vb.x; b[1] = vb.y; b[2] = vb.z; b[3] = vb.w;
    } else {
      const uint2 ra = *reinterpret_cast<const uint2 *>(x), rb = *reinterpret_cast<const uint2 *>(x + half);
      a[0] = __uint_as_float(ra.x << 16); a[1] = __uint_as_float(ra.x & 0xffff0000u);
      a[2] = __uint_as_float(ra.y << 16); a[3] = __uint_as_float(ra.y & 0xffff0000u);
      b[0] = __uint_as_float(rb.x << 16); b[1] = __uint_as_float(rb.x & 0xffff0000u);
      b[2] = __uint_as_float(rb.y << 16); b[3] = __uint_as_float(rb.y & 0xffff0000u);
    }
    const float2 *t = tab + pos * half + i;
    float ya[4], yb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float2 cs = t[j];
      ya[j] = a[j] * cs.x - b[j] * cs.y;
      yb[j] = b[j] * cs.x + a[j] * cs.y;
    }
    if constexpr (sizeof(T) == 4) {
      *reinterpret_cast<float4 *>(x) = make_float4(ya[0], ya[1], ya[2], ya[3]);
      *reinterpret_cast<float4 *>(x + half) = make_float4(yb[0], yb[1], yb[2], yb[3]);
    } else {
      bf16x4 oa, ob;
#pragma unroll
      for (int j = 0; j < 4; ++j) { oa[j] = (bf16)ya[j]; ob[j] = (bf16)yb[j]; }
      *reinterpret_cast<bf16x4 *>(x) = oa;
      *reinterpret_cast<bf16x4 *>(x + half) = ob;
    }
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

hipError_t launch_prefill_rope_table(float *tab, int n_pos, int head_dim, double base, hipStream_t s) {
  if (n_pos <= 0) return hipSuccess;
  if (head_dim % 8 || !(base > 1.0)) return hipErrorInvalidValue;
  const int half = head_dim / 2;
  hipLaunchKernelGGL(rope_table_kernel, dim3(grid_for((int64_t)n_pos * half)), dim3(256), 0, s,
                     reinterpret_cast<float2 *>(tab), n_pos, half, std::log2(base));
  return hipGetLastError();
}

hipError_t launch_prefill_rope(const PrefillJob *jobs, const int32_t *row_job, int64_t M, void *qkv, int ldqkv,
                               int nheads, int head_dim, bool bf16_mode, const float *tab, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (head_dim % 8 || ldqkv % 4) return hipErrorInvalidValue;
  const int half = head_dim / 2;
  const int grid = grid_for(M * nheads * (half / 4));
  const float2 *t = reinterpret_cast<const float2 *>(tab);
  if (bf16_mode)
    hipLaunchKernelGGL(rope_apply_kernel<bf16>, dim3(grid), dim3(256), 0, s, jobs, row_job, M, (bf16 *)qkv,
                       (int64_t)ldqkv, nheads, half, t);
  else
    hipLaunchKernelGGL(rope_apply_kernel<float>, dim3(grid), dim3(256), 0, s, jobs, row_job, M, (float *)qkv,
                       (int64_t)ldqkv, nheads, half, t);
  return hipGetLastError();
}

}  // namespace rosa
