// Time conditioning: flow time tau -> modulation table.
//
// A call needs the modulation vectors only for its distinct flow times
// (tau = k/K over the requests' step counts), so they are computed once per
// distinct tau and looked up per row afterwards.  The weights of this stage
// (two d x d time-MLP matrices and L+1 modulation projections, about 0.23 GB in
// bf16 for the pi0 shape) are streamed once per call for all distinct taus
// together: the kernel is HBM-bound on weight bytes.
#include <algorithm>

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

// Y[t][col] = act(sum_k X[t][k] W[k][col] + b[col]) for up to 16 rows t per
// pass.  A thread owns two adjacent columns: the wave reads 256 contiguous
// bytes of a weight row per k (bf16) and uses each weight for all rows.  X
// is staged in LDS transposed ([k][t]), so the 16 row values of one k are four
// broadcast 16-byte LDS reads.  The kernel is bound by streaming W once; to
// keep enough bytes in flight each thread issues 16 weight loads at a time
// and K is split over blockIdx.z, the slices' partial sums being added in
// slice order by small_gemv_reduce_kernel (deterministic).
constexpr int kGemvChunk = 128;
constexpr int kGemvRows = 16;
template <typename WT>
__global__ void __launch_bounds__(256) small_gemv_kernel(const float *__restrict__ X, int n, int K,
                                                         const WT *__restrict__ W, int N,
                                                         int k_per_slice, float *__restrict__ P) {
  constexpr int NT = kGemvRows;
  __shared__ __attribute__((aligned(16))) float xs[kGemvChunk][NT];
  const int col = 2 * (blockIdx.x * 256 + threadIdx.x);
  const int kb = blockIdx.z * k_per_slice, ke = min(K, kb + k_per_slice);
  float acc0[NT], acc1[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc0[t] = acc1[t] = 0.f;
  const WT *Wp = W + min(col, N - 2);
  for (int k0 = kb; k0 < ke; k0 += kGemvChunk) {
    const int kn = min(kGemvChunk, ke - k0);
    __syncthreads();
    for (int i = threadIdx.x; i < kn * NT; i += 256) {
      const int kk = i / NT, t = i % NT;
      xs[kk][t] = t < n ? X[(size_t)t * K + k0 + kk] : 0.f;
    }
    __syncthreads();
    for (int kk0 = 0; kk0 < kn; kk0 += 16) {
      float w0[16], w1[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int kk = min(kk0 + u, kn - 1);
        if constexpr (sizeof(WT) == 2) {
          const uint32_t v = *reinterpret_cast<const uint32_t *>(Wp + (size_t)(k0 + kk) * N);
          w0[u] = __uint_as_float(v << 16);
          w1[u] = __uint_as_float(v & 0xffff0000u);
        } else {
          const float2 f = *reinterpret_cast<const float2 *>(Wp + (size_t)(k0 + kk) * N);
          w0[u] = f.x;
          w1[u] = f.y;
        }
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        if (kk0 + u < kn) {
          const float4 *xr = reinterpret_cast<const float4 *>(&xs[kk0 + u][0]);
#pragma unroll
          for (int q = 0; q < NT / 4; ++q) {
            const float4 xv = xr[q];
            acc0[4 * q + 0] = fmaf(xv.x, w0[u], acc0[4 * q + 0]); acc1[4 * q + 0] = fmaf(xv.x, w1[u], acc1[4 * q + 0]);
            acc0[4 * q + 1] = fmaf(xv.y, w0[u], acc0[4 * q + 1]); acc1[4 * q + 1] = fmaf(xv.y, w1[u], acc1[4 * q + 1]);
            acc0[4 * q + 2] = fmaf(xv.z, w0[u], acc0[4 * q + 2]); acc1[4 * q + 2] = fmaf(xv.z, w1[u], acc1[4 * q + 2]);
            acc0[4 * q + 3] = fmaf(xv.w, w0[u], acc0[4 * q + 3]); acc1[4 * q + 3] = fmaf(xv.w, w1[u], acc1[4 * q + 3]);
          }
        }
      }
    }
  }
  if (col >= N) return;               // N is even
  float *Pz = P + (size_t)blockIdx.z * n * N;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    if (t < n) {
      Pz[(size_t)t * N + col] = acc0[t];
      Pz[(size_t)t * N + col + 1] = acc1[t];
    }
  }
}

// Y[t][col] = act(sum over slices z in order of P[z][t][col] + b[col]).
__global__ void small_gemv_reduce_kernel(const float *__restrict__ P, int slices, int n, int N,
                                         const float *__restrict__ b, int act, float *__restrict__ Y) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (size_t)n * N) return;
  float v = P[i];
  for (int z = 1; z < slices; ++z) v += P[(size_t)z * n * N + i];
  v += b ? b[i % N] : 0.f;
  if (act == 1) v = silu_f(v);
  Y[i] = v;
}

size_t small_gemv_workspace_floats(int N) { return (size_t)kGemvMaxSlices * kGemvRows * N; }

hipError_t launch_small_gemv(const float *X, int n, int K, const void *W, bool w_bf16, const float *b,
                             int N, int act, float *Y, float *ws, hipStream_t s) {
  if (N % 2) return hipErrorInvalidValue;
  for (int t0 = 0; t0 < n; t0 += kGemvRows) {
    const int nt = std::min(kGemvRows, n - t0);
    const int cols = (N / 2 + 255) / 256;
    // Enough blocks to keep ~1000 in flight, each slice at least one chunk of K.
    const int want = std::max(1, std::min((1024 + cols - 1) / cols, kGemvMaxSlices));
    const int kps = ((K + want - 1) / want + kGemvChunk - 1) / kGemvChunk * kGemvChunk;
    const int slices = (K + kps - 1) / kps;
    dim3 grid(cols, 1, slices);
    if (w_bf16)
      hipLaunchKernelGGL(small_gemv_kernel<bf16>, grid, dim3(256), 0, s, X + (size_t)t0 * K, nt, K,
                         (const bf16 *)W, N, kps, ws);
    else
      hipLaunchKernelGGL(small_gemv_kernel<float>, grid, dim3(256), 0, s, X + (size_t)t0 * K, nt, K,
                         (const float *)W, N, kps, ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t total = (size_t)nt * N;
    hipLaunchKernelGGL(small_gemv_reduce_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, ws, slices,
                       nt, N, b, act, Y + (size_t)t0 * N);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace rosa
