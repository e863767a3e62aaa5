// Per-row kernels of the action expert: batch setup (noise gather and the
// row -> modulation-row map), input projection, modulated RMSNorm, and the
// final modulated RMSNorm + velocity head + Euler update.
//
// All are HBM/L2-bound streaming kernels over the stacked action-token rows;
// one 64-lane wavefront owns one row so that the RMS reduction is a single
// wave reduction with no block barrier.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "rosa_device.h"
#include "rosa_internal.h"

namespace rosa {

// One block per request: copy its Euler state into x (the noise for a fresh
// request, else the state a previous call left in its actions), record the
// owning request of each of its rows, and for every step j < S_r of this call
// the row of the modulation table that holds tau = (k0_r + j) / K_r.
__global__ void setup_rows_kernel(const ReqDesc *__restrict__ reqs, const int32_t *__restrict__ tau_idx,
                                  int n_req, int A, int32_t *__restrict__ row_req,
                                  int32_t *__restrict__ rowmod, int M0, float *__restrict__ x) {
  const int r = blockIdx.x;
  const ReqDesc q = reqs[r];
  const float *x0 = q.k0 == 0 ? q.noise : q.actions;
  for (int i = threadIdx.x; i < q.H * A; i += blockDim.x) x[(size_t)q.tok_off * A + i] = x0[i];
  for (int t = threadIdx.x; t < q.H; t += blockDim.x) row_req[q.tok_off + t] = r;
  for (int i = threadIdx.x; i < q.H * q.S; i += blockDim.x) {
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

// h[m][n] = sum_a x[m][a] w_in[a][n] + b_in[n]   (fp32; A <= 64 is small).
// A block covers 16 rows x 256 columns: the rows of x are staged in LDS
// (broadcast reads) and each thread keeps its column of W_in in registers.
constexpr int kInProjRows = 16;
__global__ void __launch_bounds__(256) in_proj_kernel(const float *__restrict__ x, int M, int A,
                                                      const float *__restrict__ w_in,
                                                      const float *__restrict__ b_in, int d,
                                                      float *__restrict__ h) {
  __shared__ float xs[kInProjRows][64];
  const int m0 = blockIdx.y * kInProjRows;
  const int rows = min(kInProjRows, M - m0);
  for (int i = threadIdx.x; i < kInProjRows * 64; i += 256) {
    const int r = i / 64, a = i % 64;
    xs[r][a] = (r < rows && a < A) ? x[(size_t)(m0 + r) * A + a] : 0.f;
  }
  __syncthreads();
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= d) return;
  float w[64];
#pragma unroll
  for (int a = 0; a < 64; ++a) w[a] = a < A ? w_in[(size_t)a * d + n] : 0.f;
  const float bias = b_in[n];
  for (int r = 0; r < rows; ++r) {
    float acc = bias;
#pragma unroll
    for (int a = 0; a < 64; ++a) acc = fmaf(xs[r][a], w[a], acc);
    h[(size_t)(m0 + r) * d + n] = acc;
  }
}

hipError_t launch_in_proj(const float *x, int M, int A, const float *w_in, const float *b_in, int d,
                          float *h, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  dim3 grid((d + 255) / 256, (M + kInProjRows - 1) / kInProjRows);
  hipLaunchKernelGGL(in_proj_kernel, grid, dim3(256), 0, s, x, M, A, w_in, b_in, d, h);
  return hipGetLastError();
}

// u = h / sqrt(mean(h^2) + eps) * (1 + scale) + shift, with (shift, scale)
// taken from the modulation-table row of the row's flow time.  One wave per
// row; the row is read once into registers (d <= 4096: at most 16 float4 per
// lane), reduced, and written as 4-element vectors.
template <typename OutT>
__device__ __forceinline__ void store4(OutT *p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void store4<bf16>(bf16 *p, float a, float b, float c, float d) {
  bf16x4 v;
  v[0] = (bf16)a; v[1] = (bf16)b; v[2] = (bf16)c; v[3] = (bf16)d;
  *reinterpret_cast<bf16x4 *>(p) = v;
}
template <>
__device__ __forceinline__ void store4<float>(float *p, float a, float b, float c, float d) {
  *reinterpret_cast<float4 *>(p) = make_float4(a, b, c, d);
}

constexpr int kNormChunks = 16;   // float4 per lane for d = 4096
template <typename OutT, int NC>
__global__ void __launch_bounds__(256) modnorm_kernel(const float *__restrict__ h, int M, int d, float eps,
                                                      const float *__restrict__ modtab, int mod_stride,
                                                      int shift_off, int scale_off,
                                                      const int32_t *__restrict__ rowmod,
                                                      OutT *__restrict__ u, int u_rows) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= M) return;
  // The row's modulation index first; for rows of up to 1024 values its shift
  // and scale loads are also issued with the row's own loads (wider rows would
  // need so many registers that fewer waves fit).
  constexpr bool kEarlyMod = NC <= 4;
  const float *mrow = modtab + (size_t)rowmod[row] * mod_stride;
  const float *shift = mrow + shift_off;
  const float *scale = mrow + scale_off;
  const float *hr = h + (size_t)row * d;
  float4 v[NC], sc[kEarlyMod ? NC : 1], sh[kEarlyMod ? NC : 1];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int i = c * 256 + lane * 4;
    if (i < d) {
      v[c] = *reinterpret_cast<const float4 *>(hr + i);
      if constexpr (kEarlyMod) {
        sc[c] = *reinterpret_cast<const float4 *>(scale + i);
        sh[c] = *reinterpret_cast<const float4 *>(shift + i);
      }
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int i = c * 256 + lane * 4;
    if (i < d) ss += v[c].x * v[c].x + v[c].y * v[c].y + v[c].z * v[c].z + v[c].w * v[c].w;
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / (float)d + eps);
  OutT *ur = u + (size_t)row * d;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int i = c * 256 + lane * 4;
    if (i < d) {
      float4 a, b;
      if constexpr (kEarlyMod) {
        a = sc[c];
        b = sh[c];
      } else {
        a = *reinterpret_cast<const float4 *>(scale + i);
        b = *reinterpret_cast<const float4 *>(shift + i);
      }
      // row-major, or (u_rows > 0) kb32: the 4 values stay inside one 32-wide block
      OutT *up = u_rows > 0 ? u + kb32_offset(u_rows, row, i) : ur + i;
      store4<OutT>(up, v[c].x * r * (1.0f + a.x) + b.x, v[c].y * r * (1.0f + a.y) + b.y,
                   v[c].z * r * (1.0f + a.z) + b.z, v[c].w * r * (1.0f + a.w) + b.w);
    }
  }
}

hipError_t launch_modnorm(const float *h, int M, int d, float eps, const float *modtab, int mod_stride,
                          int shift_off, int scale_off, const int32_t *rowmod, void *u, bool bf16_out,
                          hipStream_t s, int u_rows) {
  if (M <= 0) return hipSuccess;
  if (d % 4 || d > kNormChunks * 256) return hipErrorInvalidValue;
  if (u_rows > 0 && (!bf16_out || d % 32 || u_rows < M)) return hipErrorInvalidValue;
  dim3 grid((M + 3) / 4);
  const int nc = (d + 255) / 256;
  auto go = [&](auto tag) {
    constexpr int NC = decltype(tag)::value;
    if (bf16_out)
      hipLaunchKernelGGL((modnorm_kernel<bf16, NC>), grid, dim3(256), 0, s, h, M, d, eps, modtab, mod_stride,
                         shift_off, scale_off, rowmod, (bf16 *)u, u_rows);
    else
      hipLaunchKernelGGL((modnorm_kernel<float, NC>), grid, dim3(256), 0, s, h, M, d, eps, modtab, mod_stride,
                         shift_off, scale_off, rowmod, (float *)u, 0);
  };
  if (nc <= 1) go(std::integral_constant<int, 1>{});
  else if (nc <= 2) go(std::integral_constant<int, 2>{});
  else if (nc <= 4) go(std::integral_constant<int, 4>{});
  else if (nc <= 8) go(std::integral_constant<int, 8>{});
  else go(std::integral_constant<int, 16>{});
  return hipGetLastError();
}

// bf16 row-major [M][K] -> kb32 planes of R rows: one thread per 8 values
// (16 bytes), consecutive threads along K within a row.
__global__ void __launch_bounds__(256) kb32_pack_kernel(const bf16 *__restrict__ src, int M, int K, int lda,
                                                        bf16 *__restrict__ dst, int R) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  const int per_row = K / 8;
  if (i >= (size_t)M * per_row) return;
  const int m = (int)(i / per_row), k = (int)(i % per_row) * 8;
  *reinterpret_cast<bf16x8 *>(dst + kb32_offset(R, m, k)) =
      *reinterpret_cast<const bf16x8 *>(src + (size_t)m * lda + k);
}

hipError_t launch_kb32_pack(const void *src, int M, int K, int lda, void *dst, int R, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (K % 32 || R < M || lda < K) return hipErrorInvalidValue;
  const size_t n = (size_t)M * (K / 8);
  hipLaunchKernelGGL(kb32_pack_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, (const bf16 *)src, M, K,
                     lda, (bf16 *)dst, R);
  return hipGetLastError();
}

// Final modulated RMSNorm, velocity v = norm W_out + b_out, Euler step
// x += (1/K_r) v, and on the request's last step of this call the store of x into the
// caller's action chunk.
//
// A block takes groups of R rows (R = 256 / A_pad, A_pad = 32 or 64): its
// waves normalize the group's rows into LDS, then each thread owns one
// (row, output) pair and walks d against W_out in LDS.  When W_out fits next
// to the rows (d * A_pad + R * d floats <= 160 KB; 128 KB + 32 KB at the pi0
// shape) it is loaded once per block and the blocks walk the row groups
// persistently; otherwise it is staged in chunks of kFinalChunk rows.
constexpr int kFinalChunk = 128;
constexpr size_t kLdsMax = 160 * 1024;
__global__ void __launch_bounds__(256) final_euler_kernel(
    const float *__restrict__ h, int M, int d, float eps, const float *__restrict__ modtab,
    int mod_stride, int shift_off, int scale_off, const int32_t *__restrict__ rowmod,
    const float *__restrict__ w_out, const float *__restrict__ b_out, int A,
    const int32_t *__restrict__ row_req, const ReqDesc *__restrict__ reqs, int step,
    float *__restrict__ x, int resident, int first_row) {
  extern __shared__ float lds_final[];
  const int a_pad = A <= 32 ? 32 : 64;
  const int R = 256 / a_pad;                       // rows per group
  const int wrows = resident ? d : kFinalChunk;    // rows of W_out held in LDS
  float *wc = lds_final;                           // [wrows][a_pad]
  float *hf = lds_final + (size_t)wrows * a_pad;   // [R][d]
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int my_r = tid / a_pad, my_a = tid % a_pad;
  auto load_w = [&](int c0, int cn) {
    for (int i = tid; i < cn * a_pad; i += 256) {
      const int ri = i / a_pad, ai = i % a_pad;
      wc[i] = ai < A ? w_out[(size_t)(c0 + ri) * A + ai] : 0.f;
    }
  };
  if (resident) load_w(0, d);
  const int n_groups = (M + R - 1) / R;
  for (int grp = blockIdx.x; grp < n_groups; grp += gridDim.x) {
    const int row0 = grp * R;
    __syncthreads();                               // previous group's reads of hf are done
    for (int r = wave; r < R; r += 4) {
      const int row = row0 + r;
      if (row >= M) continue;
      const float *hr = h + (size_t)row * d;
      float ss = 0.f;
      for (int i = lane; i < d; i += 64) ss += hr[i] * hr[i];
      ss = wave_sum(ss);
      const float rn = 1.0f / sqrtf(ss / (float)d + eps);
      const float *mrow = modtab + (size_t)rowmod[row] * mod_stride;
      for (int i = lane; i < d; i += 64)
        hf[(size_t)r * d + i] = hr[i] * rn * (1.0f + mrow[scale_off + i]) + mrow[shift_off + i];
    }
    float acc = 0.f;
    const float *hrow = hf + (size_t)my_r * d;
    if (resident) {
      __syncthreads();
      for (int i = 0; i < d; ++i) acc = fmaf(hrow[i], wc[i * a_pad + my_a], acc);
    } else {
      for (int c0 = 0; c0 < d; c0 += kFinalChunk) {
        const int cn = min(kFinalChunk, d - c0);
        __syncthreads();                           // hf written / previous chunk consumed
        load_w(c0, cn);
        __syncthreads();
        for (int i = 0; i < cn; ++i) acc = fmaf(hrow[c0 + i], wc[i * a_pad + my_a], acc);
      }
    }
    const int row = row0 + my_r;
    if (row < M && my_a < A) {
      const ReqDesc q = reqs[row_req[row]];
      const float v = acc + b_out[my_a];
      const float xn = x[(size_t)row * A + my_a] + (1.0f / (float)q.K) * v;
      x[(size_t)row * A + my_a] = xn;
      if (step == q.S - 1) q.actions[(size_t)(first_row + row - q.tok_off) * A + my_a] = xn;
    }
  }
}

hipError_t launch_final_euler(const float *h, int M, int d, float eps, const float *modtab,
                              int mod_stride, int shift_off, int scale_off, const int32_t *rowmod,
                              const float *w_out, const float *b_out, int A, const int32_t *row_req,
                              const ReqDesc *reqs, int step, float *x, int row0, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  const int a_pad = A <= 32 ? 32 : 64;
  const int R = 256 / a_pad;
  const int groups = (M + R - 1) / R;
  const size_t lds_res = ((size_t)d * a_pad + (size_t)R * d) * sizeof(float);
  const int resident = lds_res <= kLdsMax ? 1 : 0;
  const size_t lds = resident ? lds_res : ((size_t)kFinalChunk * a_pad + (size_t)R * d) * sizeof(float);
  if (lds > kLdsMax) return hipErrorInvalidValue;
  static std::atomic<bool> lds_raised{false};   // the attribute is per function: raise it to the maximum once
  if (!lds_raised.load(std::memory_order_acquire)) {
    const hipError_t e = hipFuncSetAttribute((const void *)final_euler_kernel,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsMax);
    if (e != hipSuccess) return e;
    lds_raised.store(true, std::memory_order_release);
  }
  // Resident: one block per CU walks the groups (W_out is loaded once per block).
  const int blocks = resident ? std::min(groups, 256) : std::min(groups, 1024);
  hipLaunchKernelGGL(final_euler_kernel, dim3(blocks), dim3(256), lds, s, h, M, d, eps, modtab, mod_stride,
                     shift_off, scale_off, rowmod, w_out, b_out, A, row_req, reqs, step, x, resident, row0);
  return hipGetLastError();
}

// ------------------------------------------------------------------ output projection + Euler (bf16)
// v = u W_out + b_out on the final-normalized rows u (bf16, from modnorm), then
// x += v / K and, on the request's last step of this call, x is written to its
// actions.  One block per 32-row block of u; its four waves take a quarter of
// K (= d) each, loading their quarter of the rows' u (A operand) and of W_out^T
// (B operand, bf16 [A][d], rows past A read as zero) straight into registers,
// kOutKS k-steps at a time with every load issued before the first MFMA
// (v_mfma_f32_32x32x16_bf16, NB blocks of 32 outputs).  The four partial
// products meet in LDS and are summed in wave order.  The Euler update's
// inputs (each output's request and state) are loaded before the products.
constexpr int kOutKS = 16;
template <int NB>
__global__ void __launch_bounds__(256) out_proj_euler_kernel(const bf16 *__restrict__ u, int M, int d,
                                                             const bf16 *__restrict__ wt, const float *__restrict__ b_out,
                                                             int A, const int32_t *__restrict__ row_req,
                                                             const ReqDesc *__restrict__ reqs, int step,
                                                             float *__restrict__ x, int row0, int u_rows) {
  __shared__ float part[4][NB][32 * 32];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5, l32 = lane & 31;
  const int rb = blockIdx.x;
  const int arow = min(rb * 32 + l32, M - 1);
  const int kq = d / 4, kbeg = wave * kq, kend = kbeg + kq;
  // Outputs e = tid + 256 i of the block's 32 x 32 NB: their requests' step
  // count, steps of this call and first row, and the current state.
  constexpr int NE = NB * 4;
  float xv[NE], invk[NE];
  int last[NE], arow0[NE];
  float *act[NE];
#pragma unroll
  for (int i = 0; i < NE; ++i) {
    const int e = tid + 256 * i, row = rb * 32 + ((e & 1023) >> 5), col = (e >> 10) * 32 + (e & 31);
    xv[i] = 0.f; invk[i] = 0.f; last[i] = 0; arow0[i] = 0; act[i] = nullptr;
    if (col < A && row < M) {
      const ReqDesc *q = reqs + row_req[row];
      xv[i] = x[(size_t)row * A + col];
      invk[i] = 1.0f / (float)q->K;
      last[i] = step == q->S - 1;
      arow0[i] = row0 + row - q->tok_off;
      act[i] = q->actions;
    }
  }
  f32x16 acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[nb][r] = 0.f;
  for (int k0 = kbeg; k0 < kend; k0 += 16 * kOutKS) {
    bf16x8 af[kOutKS], bfr[NB][kOutKS];
#pragma unroll
    for (int j = 0; j < kOutKS; ++j) {
      const int k = k0 + 16 * j + 8 * half;                 // 8 values inside one 32-wide block
      const bool in = k0 + 16 * j < kend;
      af[j] = in ? *reinterpret_cast<const bf16x8 *>(u + (u_rows > 0 ? kb32_offset(u_rows, arow, k) : (size_t)arow * d + k))
                 : bf16x8{};
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int col = nb * 32 + l32;
        bfr[nb][j] = in && col < A ? *reinterpret_cast<const bf16x8 *>(wt + (size_t)col * d + k) : bf16x8{};
      }
    }
#pragma unroll
    for (int j = 0; j < kOutKS; ++j)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[j], bfr[nb][j], acc[nb], 0, 0, 0);
  }
  // Lane holds output column nb 32 + lane % 32 of rows (r/4) 8 + 4 half + r%4.
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int r = 0; r < 16; ++r) part[wave][nb][((r >> 2) * 8 + half * 4 + (r & 3)) * 32 + l32] = acc[nb][r];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < NE; ++i) {
    const int e = tid + 256 * i, row = rb * 32 + ((e & 1023) >> 5), col = (e >> 10) * 32 + (e & 31);
    if (col >= A || row >= M) continue;
    const float *pp = &part[0][0][0] + e;
    const float sum = ((pp[0] + pp[NB * 1024]) + pp[2 * NB * 1024]) + pp[3 * NB * 1024];
    const float v = sum + b_out[col];
    const float xn = xv[i] + invk[i] * v;
    x[(size_t)row * A + col] = xn;
    if (last[i]) act[i][(size_t)arow0[i] * A + col] = xn;
  }
}

hipError_t launch_out_proj_euler(const bf16 *u, int M, int d, const bf16 *wt, const float *b_out, int A,
                                 const int32_t *row_req, const ReqDesc *reqs, int step, float *x, int row0,
                                 hipStream_t s, int u_rows) {
  if (M <= 0) return hipSuccess;
  if (d % 128 || A < 1 || A > 64 || (u_rows > 0 && u_rows < M)) return hipErrorInvalidValue;
  const int nrb = (M + 31) / 32;
  if (A <= 32)
    hipLaunchKernelGGL(out_proj_euler_kernel<1>, dim3(nrb), dim3(256), 0, s, u, M, d, wt, b_out, A, row_req, reqs,
                       step, x, row0, u_rows);
  else
    hipLaunchKernelGGL(out_proj_euler_kernel<2>, dim3(nrb), dim3(256), 0, s, u, M, d, wt, b_out, A, row_req, reqs,
                       step, x, row0, u_rows);
  return hipGetLastError();
}

}  // namespace rosa
