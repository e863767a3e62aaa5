// Projections of the action expert over the stacked action tokens of the
// whole batch: C[M][N] = A[M][K] W with W stored transposed ([N][K], K
// contiguous) so that both MFMA operands are K-contiguous 16-byte loads.
//
// Epilogues fuse what follows each projection: plain store (QKV), tanh-GELU
// (MLP up), and the gated residual h += gate * C whose gate row is the
// row's flow-time modulation (attention output and MLP down).
#include "rosa_device.h"
#include "rosa_internal.h"

namespace rosa {

template <int EPI, typename OutT>
__device__ __forceinline__ void epilogue_one(const GemmArgs &g, int row, int col, float v) {
  if constexpr (EPI == kEpiStore) {
    reinterpret_cast<OutT *>(g.out)[(size_t)row * g.ldo + col] = from_f32<OutT>(v);
  } else if constexpr (EPI == kEpiGelu) {
    reinterpret_cast<OutT *>(g.out)[(size_t)row * g.ldo + col] = from_f32<OutT>(gelu_tanh_f(v));
  } else {
    const float gate = g.gate[(size_t)g.rowmod[row] * g.gate_stride + col];
    float *h = reinterpret_cast<float *>(g.out) + (size_t)row * g.ldo + col;
    *h = *h + gate * v;
  }
}

// ------------------------------------------------------------------ bf16 MFMA GEMM
// Block tile 128 x 128 x 64, four waves in a 2 x 2 grid, each wave 64 x 64 =
// 2 x 2 tiles of v_mfma_f32_32x32x16_bf16.  Global -> registers -> LDS with two
// LDS buffers: the next K tile is fetched while the current one is consumed.
// LDS rows are padded by 16 bytes so that the 16-byte operand reads of 16
// consecutive rows fall in distinct banks.
namespace gb {
constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LDSW = BK + 8;   // bf16 elements per LDS row
}

template <int EPI>
__global__ void __launch_bounds__(256) gemm_bf16_kernel(GemmArgs g) {
  using namespace gb;
  __shared__ __attribute__((aligned(16))) bf16 As[2][BM * LDSW];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN * LDSW];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const bf16 *A = reinterpret_cast<const bf16 *>(g.a);
  const bf16 *W = reinterpret_cast<const bf16 *>(g.wt);

  uint4 ra[4], rb[4];
  auto load_tile = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + 256 * i, row = c >> 3, c8 = (c & 7) * 8;
      const int am = m0 + row, bn = n0 + row;
      ra[i] = am < g.M ? *reinterpret_cast<const uint4 *>(A + (size_t)am * g.lda + k0 + c8)
                       : make_uint4(0, 0, 0, 0);
      rb[i] = bn < g.N ? *reinterpret_cast<const uint4 *>(W + (size_t)bn * g.K + k0 + c8)
                       : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + 256 * i, row = c >> 3, c8 = (c & 7) * 8;
      *reinterpret_cast<uint4 *>(&As[buf][row * LDSW + c8]) = ra[i];
      *reinterpret_cast<uint4 *>(&Bs[buf][row * LDSW + c8]) = rb[i];
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = g.K / BK;
  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_tile((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 a[2], b[2];
      const int kk = ks * 16 + (lane >> 5) * 8;
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const bf16x8 *>(&As[cur][(wm * 64 + i * 32 + (lane & 31)) * LDSW + kk]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[j] = *reinterpret_cast<const bf16x8 *>(&Bs[cur][(wn * 64 + j * 32 + (lane & 31)) * LDSW + kk]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) store_tile(cur ^ 1);
    __syncthreads();
  }

  // 32x32 accumulator layout: lane l, register r -> row (r/4)*8 + (l/32)*4 + r%4, column l%32.
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn * 64 + j * 32 + (lane & 31);
      if (col >= g.N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        if (row < g.M) epilogue_one<EPI, bf16>(g, row, col, acc[i][j][r]);
      }
    }
}

// ------------------------------------------------------------------ fp32 VALU GEMM (debug mode)
// Block tile 64 x 64 x 16, each thread a 4 x 4 register tile.
template <int EPI>
__global__ void __launch_bounds__(256) gemm_f32_kernel(GemmArgs g) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const float *A = reinterpret_cast<const float *>(g.a);
  const float *W = reinterpret_cast<const float *>(g.wt);
  float acc[4][4] = {};
  const int lrow = tid >> 2, lk = (tid & 3) * 4;
  for (int k0 = 0; k0 < g.K; k0 += BK) {
    const int am = m0 + lrow, bn = n0 + lrow;
    const float4 va = am < g.M ? *reinterpret_cast<const float4 *>(A + (size_t)am * g.lda + k0 + lk)
                               : make_float4(0.f, 0.f, 0.f, 0.f);
    const float4 vb = bn < g.N ? *reinterpret_cast<const float4 *>(W + (size_t)bn * g.K + k0 + lk)
                               : make_float4(0.f, 0.f, 0.f, 0.f);
    As[lk + 0][lrow] = va.x; As[lk + 1][lrow] = va.y; As[lk + 2][lrow] = va.z; As[lk + 3][lrow] = va.w;
    Bs[lk + 0][lrow] = vb.x; Bs[lk + 1][lrow] = vb.y; Bs[lk + 2][lrow] = vb.z; Bs[lk + 3][lrow] = vb.w;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < BK; ++k) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[k][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[k][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= g.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx * 4 + j;
      if (col < g.N) epilogue_one<EPI, float>(g, row, col, acc[i][j]);
    }
  }
}

hipError_t launch_gemm(const GemmArgs &g, bool bf16_mode, hipStream_t s) {
  if (g.M <= 0) return hipSuccess;
  if (bf16_mode) {
    dim3 grid((g.N + gb::BN - 1) / gb::BN, (g.M + gb::BM - 1) / gb::BM);
    switch (g.epi) {
      case kEpiStore: hipLaunchKernelGGL(gemm_bf16_kernel<kEpiStore>, grid, dim3(256), 0, s, g); break;
      case kEpiGelu: hipLaunchKernelGGL(gemm_bf16_kernel<kEpiGelu>, grid, dim3(256), 0, s, g); break;
      default: hipLaunchKernelGGL(gemm_bf16_kernel<kEpiGatedResidual>, grid, dim3(256), 0, s, g); break;
    }
  } else {
    dim3 grid((g.N + 63) / 64, (g.M + 63) / 64);
    switch (g.epi) {
      case kEpiStore: hipLaunchKernelGGL(gemm_f32_kernel<kEpiStore>, grid, dim3(256), 0, s, g); break;
      case kEpiGelu: hipLaunchKernelGGL(gemm_f32_kernel<kEpiGelu>, grid, dim3(256), 0, s, g); break;
      default: hipLaunchKernelGGL(gemm_f32_kernel<kEpiGatedResidual>, grid, dim3(256), 0, s, g); break;
    }
  }
  return hipGetLastError();
}

}  // namespace rosa
