// Time conditioning: flow time tau -> modulation table.
//
// A call needs the modulation vectors only for its distinct flow times
// (tau = k/K over the requests' step counts), so they are computed once per
// distinct tau and looked up per row afterwards.  The weights of this stage
// (two d x d time-MLP matrices and L+1 modulation projections, about 0.23 GB in
// bf16 for the pi0 shape) are streamed once per call for all distinct taus
// together: the kernel is HBM-bound on weight bytes.
#include "rosa_device.h"
#include "rosa_internal.h"

namespace rosa {

// emb[t][i] = sin(1000 tau_t w_i), emb[t][half + i] = cos(1000 tau_t w_i),
// w_i = 10000^(-i/half).  Angles and sin/cos in double (the angle reaches 1000
// radians, where fp32 argument rounding alone would cost ~1e-4 absolute).
__global__ void time_embedding_kernel(const float *__restrict__ taus, int dt, float *__restrict__ emb) {
  const int t = blockIdx.y;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int half = dt / 2;
  if (i >= half) return;
  const double w = pow(10000.0, -(double)i / (double)half);
  const double a = 1000.0 * (double)taus[t] * w;
  emb[(size_t)t * dt + i] = (float)sin(a);
  emb[(size_t)t * dt + half + i] = (float)cos(a);
}

hipError_t launch_time_embedding(const float *taus, int n_tau, int dt, float *emb, hipStream_t s) {
  dim3 grid((dt / 2 + 255) / 256, n_tau);
  hipLaunchKernelGGL(time_embedding_kernel, grid, dim3(256), 0, s, taus, dt, emb);
  return hipGetLastError();
}

// Y[t][col] = act(sum_k X[t][k] W[k][col] + b[col]) for up to NT rows t per
// block row.  One thread per output column; W rows are read coalesced across
// the wave and each weight is used for all NT rows.
template <typename WT, int NT>
__global__ void __launch_bounds__(256) small_gemv_kernel(const float *__restrict__ X, int n, int K,
                                                         const WT *__restrict__ W,
                                                         const float *__restrict__ b, int N, int act,
                                                         float *__restrict__ Y) {
  const int col = blockIdx.x * 256 + threadIdx.x;
  const int t0 = blockIdx.y * NT;
  const int nt = min(NT, n - t0);
  if (col >= N) return;
  float acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = 0.f;
  const float *Xp = X + (size_t)t0 * K;
  int k = 0;
  for (; k + 4 <= K; k += 4) {
    float w[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) w[u] = to_f32(W[(size_t)(k + u) * N + col]);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if (t < nt) {
#pragma unroll
        for (int u = 0; u < 4; ++u) acc[t] = fmaf(Xp[(size_t)t * K + k + u], w[u], acc[t]);
      }
    }
  }
  for (; k < K; ++k) {
    const float w = to_f32(W[(size_t)k * N + col]);
#pragma unroll
    for (int t = 0; t < NT; ++t)
      if (t < nt) acc[t] = fmaf(Xp[(size_t)t * K + k], w, acc[t]);
  }
  const float bias = b ? b[col] : 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (t < nt) {
      float v = acc[t] + bias;
      if (act == 1) v = silu_f(v);
      Y[(size_t)(t0 + t) * N + col] = v;
    }
  }
}

hipError_t launch_small_gemv(const float *X, int n, int K, const void *W, bool w_bf16, const float *b,
                             int N, int act, float *Y, hipStream_t s) {
  constexpr int NT = 16;
  dim3 grid((N + 255) / 256, (n + NT - 1) / NT);
  if (w_bf16)
    hipLaunchKernelGGL((small_gemv_kernel<bf16, NT>), grid, dim3(256), 0, s, X, n, K,
                       (const bf16 *)W, b, N, act, Y);
  else
    hipLaunchKernelGGL((small_gemv_kernel<float, NT>), grid, dim3(256), 0, s, X, n, K,
                       (const float *)W, b, N, act, Y);
  return hipGetLastError();
}

}  // namespace rosa
