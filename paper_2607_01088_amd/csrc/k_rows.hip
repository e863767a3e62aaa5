// Per-row kernels of the action expert: batch setup (noise gather and the
// row -> modulation-row map), input projection, modulated RMSNorm, and the
// final modulated RMSNorm + velocity head + Euler update.
//
// All are HBM/L2-bound streaming kernels over the stacked action-token rows;
// one 64-lane wavefront owns one row so that the RMS reduction is a single
// wave reduction with no block barrier.
#include "rosa_device.h"
#include "rosa_internal.h"

namespace rosa {

// One block per request: copy its noise into the Euler state x, record the
// owning request of each of its rows, and for every step k < K_r the row of
// the modulation table that holds tau = k / K_r.
__global__ void setup_rows_kernel(const ReqDesc *__restrict__ reqs, const int32_t *__restrict__ tau_idx,
                                  int n_req, int A, int32_t *__restrict__ row_req,
                                  int32_t *__restrict__ rowmod, int M0, float *__restrict__ x) {
  const int r = blockIdx.x;
  const ReqDesc q = reqs[r];
  for (int i = threadIdx.x; i < q.H * A; i += blockDim.x) x[(size_t)q.tok_off * A + i] = q.noise[i];
  for (int t = threadIdx.x; t < q.H; t += blockDim.x) row_req[q.tok_off + t] = r;
  for (int i = threadIdx.x; i < q.H * q.K; i += blockDim.x) {
    const int k = i / q.H, t = i - k * q.H;
    rowmod[(size_t)k * M0 + q.tok_off + t] = tau_idx[k * n_req + r];
  }
}

hipError_t launch_setup_rows(const ReqDesc *reqs, int n_req, const int32_t *tau_idx, int max_steps,
                             int A, int32_t *row_req, int32_t *rowmod, int M0, float *x, hipStream_t s) {
  (void)max_steps;
  hipLaunchKernelGGL(setup_rows_kernel, dim3(n_req), dim3(256), 0, s, reqs, tau_idx, n_req, A, row_req,
                     rowmod, M0, x);
  return hipGetLastError();
}

// h[m][n] = sum_a x[m][a] w_in[a][n] + b_in[n]   (fp32; A is small)
__global__ void in_proj_kernel(const float *__restrict__ x, int A, const float *__restrict__ w_in,
                               const float *__restrict__ b_in, int d, float *__restrict__ h) {
  const int m = blockIdx.y;
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= d) return;
  const float *xr = x + (size_t)m * A;
  float acc = b_in[n];
  for (int a = 0; a < A; ++a) acc = fmaf(xr[a], w_in[(size_t)a * d + n], acc);
  h[(size_t)m * d + n] = acc;
}

hipError_t launch_in_proj(const float *x, int M, int A, const float *w_in, const float *b_in, int d,
                          float *h, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  dim3 grid((d + 255) / 256, M);
  hipLaunchKernelGGL(in_proj_kernel, grid, dim3(256), 0, s, x, A, w_in, b_in, d, h);
  return hipGetLastError();
}

// u = h / sqrt(mean(h^2) + eps) * (1 + scale) + shift, with (shift, scale)
// taken from the modulation-table row of the row's flow time.
template <typename OutT>
__global__ void __launch_bounds__(256) modnorm_kernel(const float *__restrict__ h, int M, int d, float eps,
                                                      const float *__restrict__ modtab, int mod_stride,
                                                      int shift_off, int scale_off,
                                                      const int32_t *__restrict__ rowmod,
                                                      OutT *__restrict__ u) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= M) return;
  const float *hr = h + (size_t)row * d;
  float ss = 0.f;
  for (int i = lane * 4; i < d; i += 256) {
    const float4 v = *reinterpret_cast<const float4 *>(hr + i);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / (float)d + eps);
  const float *mrow = modtab + (size_t)rowmod[row] * mod_stride;
  const float *shift = mrow + shift_off;
  const float *scale = mrow + scale_off;
  OutT *ur = u + (size_t)row * d;
  for (int i = lane * 4; i < d; i += 256) {
    const float4 v = *reinterpret_cast<const float4 *>(hr + i);
    const float4 sc = *reinterpret_cast<const float4 *>(scale + i);
    const float4 sh = *reinterpret_cast<const float4 *>(shift + i);
    ur[i + 0] = from_f32<OutT>(v.x * r * (1.0f + sc.x) + sh.x);
    ur[i + 1] = from_f32<OutT>(v.y * r * (1.0f + sc.y) + sh.y);
    ur[i + 2] = from_f32<OutT>(v.z * r * (1.0f + sc.z) + sh.z);
    ur[i + 3] = from_f32<OutT>(v.w * r * (1.0f + sc.w) + sh.w);
  }
}

hipError_t launch_modnorm(const float *h, int M, int d, float eps, const float *modtab, int mod_stride,
                          int shift_off, int scale_off, const int32_t *rowmod, void *u, bool bf16_out,
                          hipStream_t s) {
  if (M <= 0) return hipSuccess;
  dim3 grid((M + 3) / 4);
  if (bf16_out)
    hipLaunchKernelGGL(modnorm_kernel<bf16>, grid, dim3(256), 0, s, h, M, d, eps, modtab, mod_stride,
                       shift_off, scale_off, rowmod, (bf16 *)u);
  else
    hipLaunchKernelGGL(modnorm_kernel<float>, grid, dim3(256), 0, s, h, M, d, eps, modtab, mod_stride,
                       shift_off, scale_off, rowmod, (float *)u);
  return hipGetLastError();
}

// Final modulated RMSNorm, velocity v = norm W_out + b_out, Euler step
// x += (1/K_r) v, and on the request's last step the store of x into the
// caller's action chunk.  One wave per row; the normalized row is staged in
// LDS so that the A output dot products read it as a broadcast.
__global__ void __launch_bounds__(256) final_euler_kernel(
    const float *__restrict__ h, int M, int d, float eps, const float *__restrict__ modtab,
    int mod_stride, int shift_off, int scale_off, const int32_t *__restrict__ rowmod,
    const float *__restrict__ w_out, const float *__restrict__ b_out, int A,
    const int32_t *__restrict__ row_req, const ReqDesc *__restrict__ reqs, int step,
    float *__restrict__ x) {
  extern __shared__ float lds_rows[];  // [4][d]
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + w;
  const bool active = row < M;
  float *hf = lds_rows + (size_t)w * d;
  if (active) {
    const float *hr = h + (size_t)row * d;
    float ss = 0.f;
    for (int i = lane; i < d; i += 64) ss += hr[i] * hr[i];
    ss = wave_sum(ss);
    const float r = 1.0f / sqrtf(ss / (float)d + eps);
    const float *mrow = modtab + (size_t)rowmod[row] * mod_stride;
    for (int i = lane; i < d; i += 64) hf[i] = hr[i] * r * (1.0f + mrow[scale_off + i]) + mrow[shift_off + i];
  }
  __syncthreads();
  if (!active) return;
  const ReqDesc q = reqs[row_req[row]];
  const float dt = 1.0f / (float)q.K;
  const int half = lane >> 5;
  for (int a0 = 0; a0 < A; a0 += 32) {
    const int a = a0 + (lane & 31);
    float acc = 0.f;
    if (a < A)
      for (int i = half; i < d; i += 2) acc = fmaf(hf[i], w_out[(size_t)i * A + a], acc);
    acc += __shfl_xor(acc, 32, 64);
    if (half == 0 && a < A) {
      const float v = acc + b_out[a];
      const float xn = x[(size_t)row * A + a] + dt * v;
      x[(size_t)row * A + a] = xn;
      if (step == q.K - 1) q.actions[(size_t)(row - q.tok_off) * A + a] = xn;
    }
  }
}

hipError_t launch_final_euler(const float *h, int M, int d, float eps, const float *modtab,
                              int mod_stride, int shift_off, int scale_off, const int32_t *rowmod,
                              const float *w_out, const float *b_out, int A, const int32_t *row_req,
                              const ReqDesc *reqs, int step, float *x, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  const size_t lds = (size_t)4 * d * sizeof(float);
  hipLaunchKernelGGL(final_euler_kernel, dim3((M + 3) / 4), dim3(256), lds, s, h, M, d, eps, modtab,
                     mod_stride, shift_off, scale_off, rowmod, w_out, b_out, A, row_req, reqs, step, x);
  return hipGetLastError();
}

}  // namespace rosa
