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
// Block tile BM x BN, WM x WN waves, each wave a (BM/WM) x (BN/WN) tile made of
// 32 x 32 v_mfma_f32_32x32x16_bf16 accumulators.
//
// K is consumed 32 at a time through a ring of four LDS stages filled by
// global_load_lds_dwordx4 (global -> LDS without staging registers): while the
// waves multiply stage s, stages s+1 and s+2 are landing and stage s+3 is
// being requested.  One barrier per stage.  Each stage buffer is its own LDS
// object and the barrier is a bare s_barrier, so the only wait on the
// asynchronous copies is the explicit vmcnt before it.
//
// LDS rows are 64 bytes (32 bf16 of K); the four 16-byte chunks of row r are
// stored XOR-swizzled by (r / 4) % 4, so the 16 rows a 16-lane group reads at
// one logical chunk land in 16 distinct bank groups.  The copy writes lane i
// of a wave's instruction to byte 16 i of a 1 KB block (16 rows), so each
// lane fetches the logical chunk that belongs at its physical position.
namespace gb {
constexpr int BK = 32;
constexpr int NST = 4;
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
}  // namespace gb

#define ROSA_LDS(p) ((__attribute__((address_space(3))) void *)(p))

template <int BM_, int BN_, int WM_, int WN_>
struct GemmTile {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, NW = WM_ * WN_, NT = 64 * NW;
  static constexpr int TM = BM / WM / 32, TN = BN / WN / 32;     // MFMA tiles per wave
  static constexpr int ABYTES = BM * gb::BK * 2, SBYTES = ABYTES + BN * gb::BK * 2;
  static constexpr int DA = BM / 16 / NW, DB = BN / 16 / NW;      // 1 KB copies per wave per stage
  static_assert(DA * 16 * NW == BM && DB * 16 * NW == BN, "copy split");
  static_assert(TM * 32 * WM == BM && TN * 32 * WN == BN, "wave split");
  static constexpr int WAIT = gb::waitcnt_vm((DA + DB) * (gb::NST - 2));
  static constexpr int WAIT0 = gb::waitcnt_vm(0);
};

template <typename T, int EPI>
__global__ void __launch_bounds__(T::NT) gemm_bf16_kernel(GemmArgs g) {
  using namespace gb;
  constexpr int ABYTES = T::ABYTES, SBYTES = T::SBYTES, DA = T::DA, DB = T::DB, TM = T::TM, TN = T::TN;
  constexpr int NW = T::NW;
  __shared__ __attribute__((aligned(1024))) uint8_t L0[SBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t L1[SBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t L2[SBYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t L3[SBYTES];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & (T::NW - 1);   // wave-uniform, in an SGPR
  const int wm = wave / T::WN, wn = wave % T::WN;
  const int m0 = blockIdx.y * T::BM, n0 = blockIdx.x * T::BN;
  const bf16 *A = reinterpret_cast<const bf16 *>(g.a);
  const bf16 *W = reinterpret_cast<const bf16 *>(g.wt);

  // Copy sources: instruction j of this wave fills rows 16 (NW j + wave) .. +15;
  // lane i writes physical chunk i % 4 of row i / 4 there, which holds logical
  // chunk (i % 4) ^ ((row / 4) % 4) = (i % 4) ^ ((i / 16) % 4).
  const int csrc = (lane & 3) ^ ((lane >> 4) & 3);
  const bf16 *asrc[DA];
  const bf16 *bsrc[DB];
#pragma unroll
  for (int j = 0; j < DA; ++j) {
    const int row = min(m0 + (NW * j + wave) * 16 + (lane >> 2), g.M - 1);
    asrc[j] = A + (size_t)row * g.lda + csrc * 8;
  }
#pragma unroll
  for (int j = 0; j < DB; ++j) {
    const int row = min(n0 + (NW * j + wave) * 16 + (lane >> 2), g.N - 1);
    bsrc[j] = W + (size_t)row * g.K + csrc * 8;
  }
  const int nk = g.K / BK;
  auto issue = [&](uint8_t *st, int kt) {
    const int k0 = min(kt, nk - 1) * BK;
#pragma unroll
    for (int j = 0; j < DA; ++j)
      __builtin_amdgcn_global_load_lds((const void *)(asrc[j] + k0), ROSA_LDS(st + (NW * j + wave) * 1024), 16, 0, 0);
#pragma unroll
    for (int j = 0; j < DB; ++j)
      __builtin_amdgcn_global_load_lds((const void *)(bsrc[j] + k0), ROSA_LDS(st + ABYTES + (NW * j + wave) * 1024),
                                       16, 0, 0);
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Operand reads: lane reads row (lane & 31) of a 32-row tile, logical chunk
  // 2 ks + lane / 32, at physical chunk (logical) ^ ((lane / 4) % 4).
  const int swz = (lane >> 2) & 3;
  const int ph0 = (lane >> 5) ^ swz, ph1 = (2 + (lane >> 5)) ^ swz;
  const int arow = (wm * TM * 32 + (lane & 31)) * 64;
  const int brow = ABYTES + (wn * TN * 32 + (lane & 31)) * 64;
  auto compute = [&](const uint8_t *st) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int ph = (ks == 0 ? ph0 : ph1) * 16;
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = *reinterpret_cast<const bf16x8 *>(st + arow + i * 32 * 64 + ph);
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[j] = *reinterpret_cast<const bf16x8 *>(st + brow + j * 32 * 64 + ph);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
  };
  auto step = [&](uint8_t *cur, uint8_t *refill, int kt) {
    __builtin_amdgcn_s_waitcnt(T::WAIT);    // this wave's copies of stage kt have landed
    __builtin_amdgcn_s_barrier();           // ... and every wave's; stage kt-1 is no longer read
    __builtin_amdgcn_sched_barrier(0);
    issue(refill, kt + NST - 1);
    compute(cur);
  };

  issue(L0, 0);
  issue(L1, 1);
  issue(L2, 2);
  for (int kt = 0; kt < nk; kt += 4) {      // nk is a multiple of 4
    step(L0, L3, kt);
    step(L1, L0, kt + 1);
    step(L2, L1, kt + 2);
    step(L3, L2, kt + 3);
  }
  __builtin_amdgcn_s_waitcnt(T::WAIT0);     // no copy may outlive the block's LDS

  // 32x32 accumulator layout: lane l, register r -> row (r/4)*8 + (l/32)*4 + r%4, column l%32.
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = n0 + wn * TN * 32 + j * 32 + (lane & 31);
      if (col >= g.N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * TM * 32 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        if (row < g.M) epilogue_one<EPI, bf16>(g, row, col, acc[i][j][r]);
      }
    }
}

using Tile256x4 = GemmTile<256, 256, 2, 2>;    // 4 waves, 128 x 128 each
using Tile256x8 = GemmTile<256, 256, 2, 4>;    // 8 waves, 128 x 64 each
using Tile256x16 = GemmTile<256, 256, 4, 4>;   // 16 waves, 64 x 64 each
using Tile128x4 = GemmTile<128, 128, 2, 2>;    // 4 waves, 64 x 64 each
using Tile256x128 = GemmTile<256, 128, 2, 2>;  // 4 waves, 128 x 64 each

template <typename T>
static hipError_t launch_tile(const GemmArgs &g, hipStream_t s) {
  dim3 grid((g.N + T::BN - 1) / T::BN, (g.M + T::BM - 1) / T::BM);
  switch (g.epi) {
    case kEpiStore: hipLaunchKernelGGL((gemm_bf16_kernel<T, kEpiStore>), grid, dim3(T::NT), 0, s, g); break;
    case kEpiGelu: hipLaunchKernelGGL((gemm_bf16_kernel<T, kEpiGelu>), grid, dim3(T::NT), 0, s, g); break;
    default: hipLaunchKernelGGL((gemm_bf16_kernel<T, kEpiGatedResidual>), grid, dim3(T::NT), 0, s, g); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm_cfg(const GemmArgs &g, int cfg, hipStream_t s) {
  if (g.M <= 0) return hipSuccess;
  if (g.K % 128 != 0) return hipErrorInvalidValue;
  switch (cfg) {
    case 0: return launch_tile<Tile256x4>(g, s);
    case 1: return launch_tile<Tile256x8>(g, s);
    case 2: return launch_tile<Tile256x16>(g, s);
    case 3: return launch_tile<Tile128x4>(g, s);
    case 4: return launch_tile<Tile256x128>(g, s);
    default: return hipErrorInvalidValue;
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
    // 256 x 256 blocks of 16 waves (one block per CU) or 128 x 128 blocks of 4
    // waves (two per CU), whichever needs less time: full rounds of blocks over
    // the CUs times the measured time of one round (per 1024 of K: 33 us for
    // 256 x 256 blocks, 19 us for 128 x 128 blocks on MI355X).  Small M with
    // N = d leaves most CUs idle with the large blocks.
    static int n_cu = 0;
    if (n_cu == 0) {
      int dev = 0, v = 0;
      if (hipGetDevice(&dev) == hipSuccess &&
          hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
        n_cu = v;
      else
        n_cu = 256;
    }
    const long t256 = (long)((g.M + 255) / 256) * ((g.N + 255) / 256);
    const long t128 = (long)((g.M + 127) / 128) * ((g.N + 127) / 128);
    const long cost256 = (t256 + n_cu - 1) / n_cu * 33;
    const long cost128 = (t128 + 2 * n_cu - 1) / (2 * n_cu) * 19;
    return launch_gemm_cfg(g, cost128 < cost256 ? 3 : 2, s);
  }
  dim3 grid((g.N + 63) / 64, (g.M + 63) / 64);
  switch (g.epi) {
    case kEpiStore: hipLaunchKernelGGL(gemm_f32_kernel<kEpiStore>, grid, dim3(256), 0, s, g); break;
    case kEpiGelu: hipLaunchKernelGGL(gemm_f32_kernel<kEpiGelu>, grid, dim3(256), 0, s, g); break;
    default: hipLaunchKernelGGL(gemm_f32_kernel<kEpiGatedResidual>, grid, dim3(256), 0, s, g); break;
  }
  return hipGetLastError();
}

}  // namespace rosa
