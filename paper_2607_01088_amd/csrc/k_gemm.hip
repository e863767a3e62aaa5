// Projections of the action expert over the stacked action tokens of the
// whole batch: C[M][N] = A[M][K] W with W stored transposed ([N][K], K
// contiguous) so that both MFMA operands are K-contiguous 16-byte loads.
//
// Epilogues fuse what follows each projection: plain store (QKV), tanh-GELU
// (MLP up), and the gated residual h += gate * C whose gate row is the
// row's flow-time modulation (attention output and MLP down).  Launches with
// few tiles (few rows) may split K over several blocks per tile: each block
// stores its slice's fp32 product (kEpiPartial) and a second kernel sums the
// slices in order and applies the epilogue.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "rosa_device.h"
#include "rosa_internal.h"

namespace rosa {

// ------------------------------------------------------------------ bf16 MFMA GEMM
// Block tile BM x BN = (32 MB) x (32 TN WN), WM x WN waves, each wave
// (32 MB / WM) x (32 TN) made of 32 x 32 v_mfma_f32_32x32x16_bf16 tiles.
//
// Main loop: K is consumed BK (32 or 64) at a time through a ring of NST = 4
// LDS stages filled by global_load_lds_dwordx4 (global -> LDS without
// staging registers): while the waves multiply stage s, stage s+1 has landed
// and stages s+2 .. s+NST-1 are landing or being requested, so NST - 2 stages
// of copies cover the memory latency.  One barrier per stage, crossed before the stage's last
// k-step of MFMAs so that the next stage's first operand reads overlap them;
// within a stage each k-step's operands are read while the previous k-step's
// MFMAs run.  The copies are issued as
// inline assembly the compiler does not track and the barrier is a bare
// s_barrier, so the only wait on them is the explicit vmcnt before it.
//
// LDS rows are 64 bytes (32 bf16 of K); the four 16-byte chunks of row r are
// stored XOR-swizzled by (r / 4) % 4, so the 16 rows a 16-lane group reads at
// one logical chunk land in 16 distinct bank groups.  A copy instruction
// writes lane i to byte 16 i of a 1 KB block (16 rows), so each lane fetches
// the logical chunk that belongs at its physical position.
//
// The MFMA takes the weight fragment as its first operand, so a lane's
// accumulator registers hold four consecutive output columns of one output row.
// The epilogue stages each 32 x 32 accumulator tile through LDS and writes
// whole 64- or 128-byte row segments with 16-byte accesses.
//
// Blocks are mapped to tiles so that each of the 8 XCDs (which receive blocks
// round-robin) works on a contiguous range of the row-major tile list: the
// column tiles of one row panel share an XCD's L2.
namespace gb {
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
// f(integral_constant<int, i>) for i = 0 .. N - 1, in order.
template <int N, int I = 0, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}
}  // namespace gb


// Chunk swizzle of an LDS row of CPR 16-byte chunks: chunk c of row r is
// stored at c ^ gswz(r).  64-byte rows (CPR 4): (r / 4) % 4; 128-byte rows
// (CPR 8): (r / 2) % 8.  Either way the 16 rows a 16-lane group reads at one
// logical chunk fall in 16 distinct bank groups.
template <int CPR>
__device__ __forceinline__ int gswz(int r) { return CPR == 4 ? (r >> 2) & 3 : (r >> 1) & 7; }

template <int MB_, int TN_, int WM_, int WN_, int BK_ = 32, int NST_ = 4>
struct GemmTile {
  static constexpr int MB = MB_, TN = TN_, WM = WM_, WN = WN_, NW = WM_ * WN_, NT = 64 * NW;
  static constexpr int MBW = MB / WM;                                   // 32-row blocks per wave
  static constexpr int BM = 32 * MB, BN = 32 * TN * WN;
  static constexpr int BK = BK_;                                        // K per stage
  static constexpr int ROWB = BK * 2, CPR = ROWB / 16, RPU = 1024 / ROWB;   // row bytes, chunks per row, rows per 1 KB
  static constexpr int ABYTES = BM * BK * 2, SBYTES = ABYTES + BN * BK * 2;
  // LDS ring depth: 4, or 8 for the 64-row tiles of small launches (one
  // block per CU, latency-bound: more copies in flight per CU).  Deeper rings
  // measured no faster on the larger tiles.
  static constexpr int NST = NST_;
  static_assert(NST * SBYTES <= 160 * 1024, "LDS");
  static constexpr int U = (BM + BN) / RPU;                             // 1 KB copies per stage
  static_assert(BK == 32 || BK == 64, "stage K");
  static constexpr int CHI = (U + NW - 1) / NW, CLO = U / NW;           // copies per wave
  static constexpr int NHI = U % NW == 0 ? NW : U % NW;                 // waves with CHI copies
  static_assert(MBW * WM == MB, "row split");
  static_assert(NW * 4096 <= NST * SBYTES, "epilogue staging space (4 KB per wave)");
};

// K stages [kt0, kt0 + nk) of the tile at (m0, n0) into acc (zeroed first).
// Ends with every copy landed and every wave past its last LDS read.
template <typename T>
__device__ __forceinline__ void gemm_mainloop(const GemmArgs &g, int m0, int n0, int kt0, int nk, uint8_t *L,
                                              f32x16 (&acc)[T::MBW][T::TN]) {
  using namespace gb;
  constexpr int NW = T::NW, MBW = T::MBW, TN = T::TN, CHI = T::CHI, CLO = T::CLO, NST = T::NST;
  constexpr int ABYTES = T::ABYTES, SBYTES = T::SBYTES;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) % NW;   // wave-uniform, in an SGPR
  const int wm = wave / T::WN, wn = wave % T::WN;
  const bf16 *A = reinterpret_cast<const bf16 *>(g.a);
  const bf16 *W = reinterpret_cast<const bf16 *>(g.wt);

  // Copy sources: 1 KB unit u (A rows first, then W rows) is copied by wave
  // u % NW; lane i writes physical chunk i % CPR of row i / CPR of the unit,
  // which holds logical chunk (i % CPR) ^ gswz(row).  Both operands are kb32
  // (planes of R rows: a_rows for A, N for W), so logical chunk c of a row
  // (k = k0 + 8 c) lies in plane k0 / 32 + c / 4 and a unit reads one (32 of
  // K) or two (64 of K) contiguous 512 B - 1 KB runs.  Rows past M (or N)
  // re-read the last row; their results are never stored.
  constexpr int CPR = T::CPR, RPU = T::RPU;
  const bf16 *src[CHI];
  size_t kstep[CHI];                        // elements per 32 of K: 32 R
#pragma unroll
  for (int j = 0; j < CHI; ++j) {
    const int u = min(j * NW + wave, T::U - 1);
    const int lrow = u * RPU + lane / CPR;                   // row within the stage
    const int csrc = (lane % CPR) ^ gswz<CPR>(lrow);
    if (u < T::BM / RPU) {
      const int row = min(m0 + lrow, g.M - 1);
      kstep[j] = (size_t)g.a_rows * 32;
      src[j] = A + ((size_t)(csrc >> 2) * g.a_rows + row) * 32 + (csrc & 3) * 8;
    } else {
      const int row = min(n0 + lrow - T::BM, g.N - 1);
      kstep[j] = (size_t)g.N * 32;
      src[j] = W + ((size_t)(csrc >> 2) * g.N + row) * 32 + (csrc & 3) * 8;
    }
  }
  const bool hi = wave < T::NHI;
  constexpr int BK = T::BK, ROWB = T::ROWB;
  // Copy j (of CHI) of this wave for stage kt into buffer st.
  auto issue_one = [&](uint8_t *st, int kt, int j) __attribute__((always_inline)) {
    const int kb = (kt0 + min(kt, nk - 1)) * (BK / 32);   // past the end: repeat the last stage (never read)
    if (j < CLO || hi) dma_1k(src[j] + (size_t)kb * kstep[j], lds_u32(st) + (uint32_t)((j * NW + wave) * 1024));
  };
  auto issue = [&](uint8_t *st, int kt) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < CHI; ++j) issue_one(st, kt, j);
  };

#pragma unroll
  for (int i = 0; i < MBW; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Operand reads: lane reads row (lane & 31) of a 32-row block, logical chunk
  // 2 ks + lane / 32, at physical chunk (logical) ^ gswz(row); every 32-row
  // block starts at a multiple of 32 rows, so the swizzle depends on lane & 31.
  constexpr int NKS = BK / 16;
  const int swz = gswz<CPR>(lane & 31);
  int ph[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) ph[ks] = ((2 * ks + (lane >> 5)) ^ swz) * 16;
  const int arow = (wm * MBW * 32 + (lane & 31)) * ROWB;
  const int brow = ABYTES + (wn * TN * 32 + (lane & 31)) * ROWB;
  // Fragments of one k-step (MBW A tiles, TN W tiles), double-buffered.
  bf16x8 fa[2][MBW], fb[2][TN];
  auto read_frags = [&](const uint8_t *st, int ks, int f) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < TN; ++j) fb[f][j] = *reinterpret_cast<const bf16x8 *>(st + brow + j * 32 * ROWB + ph[ks]);
#pragma unroll
    for (int i = 0; i < MBW; ++i) fa[f][i] = *reinterpret_cast<const bf16x8 *>(st + arow + i * 32 * ROWB + ph[ks]);
  };
  // The k-step's MFMAs; after MFMA number q, between(q) (the refill copies,
  // spread over the k-step so that no wave stalls on a burst of copies while
  // its MFMAs wait to issue).
  auto mfmas = [&](int f, auto &&between) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < MBW; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[f][j], fa[f][i], acc[i][j], 0, 0, 0);
        between(i * TN + j);
      }
  };
  constexpr int NMF = MBW * TN;            // MFMAs per k-step
  // Stage kt in buffer kt % NST (`cur`), whose k-step 0 fragments are
  // already in registers.  Each k-step first reads the next k-step's
  // fragments, then issues its own MFMAs, so LDS latency hides behind a
  // k-step of MFMAs.  Before the last k-step's MFMAs the block crosses the
  // stage boundary: wait until this wave's copies of stage kt + 1 have landed
  // (stages kt + 2 .. kt + NST - 2 may still be in flight), barrier (every
  // wave's copies have landed, and every wave has finished reading stage
  // kt - 1), refill stage kt - 1's buffer with stage kt + NST - 1, and read
  // stage kt + 1's first fragments.
  auto stage = [&](auto cur_t, int kt) __attribute__((always_inline)) {
    constexpr int cur = decltype(cur_t)::value;
    constexpr int nxt = cur + 1 == NST ? 0 : cur + 1, old = cur == 0 ? NST - 1 : cur - 1;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      if (ks + 1 < NKS) {
        read_frags(L + cur * SBYTES, ks + 1, (ks + 1) & 1);
      } else {
        if (hi) __builtin_amdgcn_s_waitcnt(waitcnt_vm((NST - 3) * CHI));
        else __builtin_amdgcn_s_waitcnt(waitcnt_vm((NST - 3) * CLO));
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        read_frags(L + nxt * SBYTES, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (ks + 1 < NKS) {
        mfmas(ks & 1, [](int) {});
      } else {
        // copy j after MFMA (j * NMF) / CHI: spread evenly over the k-step
        mfmas(ks & 1, [&](int q) __attribute__((always_inline)) {
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int j = 0; j < CHI; ++j)
            if ((j * NMF) / CHI == q) issue_one(L + old * SBYTES, kt + NST - 1, j);
          __builtin_amdgcn_sched_barrier(0);
        });
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  static_assert(NKS % 2 == 0, "the next stage's first fragments go to buffer 0");

  // Prologue: stages 0 .. NST - 2 requested, stage 0 landed.
#pragma unroll
  for (int st = 0; st < NST - 1; ++st) issue(L + st * SBYTES, st);
  if (hi) __builtin_amdgcn_s_waitcnt(waitcnt_vm((NST - 2) * CHI));
  else __builtin_amdgcn_s_waitcnt(waitcnt_vm((NST - 2) * CLO));
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  read_frags(L, 0, 0);
  // Groups of NST stages, unrolled so that every buffer offset is an
  // immediate, then the remaining stages.
  int kt = 0;
  for (; kt + NST <= nk; kt += NST)
    static_for<NST>([&](auto r) { stage(r, kt + decltype(r)::value); });
  static_for<NST - 1>([&](auto r) {
    if (kt + decltype(r)::value < nk) stage(r, kt + decltype(r)::value);
  });
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  __syncthreads();                          // every wave is past its last stage read: LDS is free
}

// Epilogue of the tile at (m0, n0) from acc; stages through the ring's LDS,
// which must be free (gemm_mainloop ends that way).  DN: the deferred norm's
// part of the epilogue (outputs t and the row sums of squares after a gated
// residual; the norm's completion before a bf16 store).
template <typename T, int EPI, bool DN = false>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs &g, int m0, int n0, uint8_t *L,
                                              f32x16 (&acc)[T::MBW][T::TN]) {
  constexpr int MBW = T::MBW, TN = T::TN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) % T::NW;
  const int wm = wave / T::WN, wn = wave % T::WN;
  // Register r of tile (i, j) holds row m0 + 32 (wm MBW + i) + lane % 32,
  // columns n0 + 32 (wn TN + j) + 8 (r / 4) + 4 (lane / 32) + r % 4: four
  // consecutive columns per 4 registers.
  const int r32 = lane & 31, half = lane >> 5;
  if constexpr (EPI == kEpiGatedResidual || EPI == kEpiPartial) {
    // h += gate[rowmod[row]] * acc (or, for a K slice, out = acc in fp32).
    // Each wave stages one 32 x 32 tile at a
    // time in its own 4 KB slot (fp32: 32 rows x 8 chunks of 16 B, chunk c of
    // row r at c ^ ((r / 2) % 8)), then reads it back row-contiguous.
    uint8_t *stg = L + wave * 4096;
    float *H = reinterpret_cast<float *>(g.out);
    // Gate rows of every row this lane touches, loaded once up front so that
    // no gate load waits for its row's modulation index (32-bit offsets: the
    // gate table has far fewer than 2^31 elements).  Tiles of 16 waves have no
    // registers to spare (128 per lane) and look the index up per use.
    constexpr bool kHoist = T::NW < 16 && EPI == kEpiGatedResidual;
    int goff[kHoist ? MBW : 1][4];
    if constexpr (kHoist) {
#pragma unroll
      for (int i = 0; i < MBW; ++i)
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const int row = min(m0 + (wm * MBW + i) * 32 + 8 * p + (lane >> 3), g.M - 1);
          goff[i][p] = g.rowmod[row] * g.gate_stride;
        }
    }
    // Pass p of 32 x 32 tile q = i TN + j: rows 8 p + lane / 8, columns
    // 4 (lane % 8) .. + 3.  The residual and gate rows of tile q + 1 are
    // requested before tile q is combined, so each tile's global loads wait
    // behind the previous tile's work instead of stalling on their own
    // (two register sets; 16-wave tiles, and tiles small enough to run two
    // blocks per CU, have no registers to spare and load each tile's rows
    // just before use).
    constexpr int Q = MBW * TN;
    constexpr bool kTwoBlocks = T::NST * T::SBYTES <= 80 * 1024;
    constexpr int NB = (EPI == kEpiGatedResidual && T::NW < 16 && !kTwoBlocks && !DN) ? 2 : 1;
    float4 hv[NB][4], gt[NB][4];
    // The deferred norm's scale rows load with the tile's other rows, except in
    // 16-wave tiles (no registers to spare), which load them at use.
    constexpr bool kScvAhead = DN && T::NW < 16;
    float4 scv[kScvAhead ? NB : 1][4];
    const int col0 = (lane & 7) * 4;
    auto load_rows = [&](int q, int buf) __attribute__((always_inline)) {
      const int i = q / TN, j = q % TN;
      const int rb = m0 + (wm * MBW + i) * 32, col = n0 + (wn * TN + j) * 32 + col0;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int row = rb + 8 * p + (lane >> 3);
        if (row < g.M && col < g.N) {
          hv[buf][p] = *reinterpret_cast<const float4 *>(H + (size_t)row * g.ldo + col);
          if constexpr (kHoist) gt[buf][p] = *reinterpret_cast<const float4 *>(g.gate + goff[i][p] + col);
          else gt[buf][p] = *reinterpret_cast<const float4 *>(g.gate + (size_t)g.rowmod[row] * g.gate_stride + col);
          if constexpr (kScvAhead) {
            if constexpr (kHoist) scv[buf][p] = *reinterpret_cast<const float4 *>(g.dscale + goff[i][p] + col);
            else scv[buf][p] = *reinterpret_cast<const float4 *>(g.dscale + (size_t)g.rowmod[row] * g.gate_stride + col);
          }
        }
      }
    };
    if constexpr (EPI == kEpiGatedResidual && NB == 2) load_rows(0, 0);
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int i = q / TN, j = q % TN, buf = NB == 2 ? (q & 1) : 0;
      if constexpr (EPI == kEpiGatedResidual) {
        if (NB == 1) load_rows(q, 0);
        else if (q + 1 < Q) load_rows(q + 1, (q + 1) & 1);
      }
      const int rb = m0 + (wm * MBW + i) * 32, col = n0 + (wn * TN + j) * 32 + col0;
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int c = (2 * gq + half) ^ ((r32 >> 1) & 7);
        *reinterpret_cast<float4 *>(stg + r32 * 128 + c * 16) =
            make_float4(acc[i][j][4 * gq], acc[i][j][4 * gq + 1], acc[i][j][4 * gq + 2], acc[i][j][4 * gq + 3]);
      }
      float4 v[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int rr = 8 * p + (lane >> 3), c = lane & 7;
        v[p] = *reinterpret_cast<const float4 *>(stg + rr * 128 + ((c ^ ((rr >> 1) & 7)) * 16));
      }
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const int row = rb + 8 * p + (lane >> 3);
        float q2 = 0.f;
        if (row < g.M && col < g.N) {
          if constexpr (EPI == kEpiPartial) {
            *reinterpret_cast<float4 *>(H + (size_t)row * g.ldo + col) = v[p];
          } else {
            float4 h = hv[buf][p];
            h.x = h.x + gt[buf][p].x * v[p].x;
            h.y = h.y + gt[buf][p].y * v[p].y;
            h.z = h.z + gt[buf][p].z * v[p].z;
            h.w = h.w + gt[buf][p].w * v[p].w;
            *reinterpret_cast<float4 *>(H + (size_t)row * g.ldo + col) = h;
            if constexpr (DN) {
              float4 sc;
              if constexpr (kScvAhead) sc = scv[buf][p];
              else sc = *reinterpret_cast<const float4 *>(g.dscale + (size_t)g.rowmod[row] * g.gate_stride + col);
              bf16x4 tv;
              tv[0] = (bf16)(h.x * (1.0f + sc.x));
              tv[1] = (bf16)(h.y * (1.0f + sc.y));
              tv[2] = (bf16)(h.z * (1.0f + sc.z));
              tv[3] = (bf16)(h.w * (1.0f + sc.w));
              *reinterpret_cast<bf16x4 *>(reinterpret_cast<bf16 *>(g.dt) + kb32_offset(g.dt_rows, row, col)) = tv;
              q2 = fmaf(h.w, h.w, fmaf(h.z, h.z, fmaf(h.y, h.y, h.x * h.x)));
            }
          }
        }
        if constexpr (DN) {
          // The row's 32 columns of this tile sit on the 8 lanes lane / 8
          // shares; their sum (fixed butterfly order) goes to the row's entry.
          q2 += __shfl_xor(q2, 1, 64);
          q2 += __shfl_xor(q2, 2, 64);
          q2 += __shfl_xor(q2, 4, 64);
          if ((lane & 7) == 0 && row < g.M && col < g.N) g.dss[(size_t)row * (g.N >> 5) + (col >> 5)] = q2;
        }
      }
    }
  } else {
    // Each wave stages one 32 x 32 tile at a time in its own 4 KB slot, then
    // reads it back row-contiguous.
    uint8_t *stg = L + wave * 4096;
    // Deferred norm: 1 / rms of this lane's row in each row block, its sum of
    // squares taken over the two lane halves (each half sums its share of the
    // row's block sums in order; the halves' totals are then added).
    // The shift rows of every column this lane stores are loaded here too, all
    // before the first store (the stores could alias them for the compiler);
    // 16-wave tiles (no registers to spare) load each 32 x 32 tile's before it.
    constexpr bool kShAll = DN && T::NW < 16;
    float rinv[DN ? MBW : 1];
    int mrow[DN ? MBW : 1];
    f32x4 shv[kShAll ? MBW : 1][kShAll ? TN : 1][4];
    auto load_shift = [&](int i, int j, f32x4 (&dst)[4]) __attribute__((always_inline)) {
      const float *shrow = g.cshift + (size_t)mrow[i] * g.cshift_stride;
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int c4 = n0 + (wn * TN + j) * 32 + 8 * gq + 4 * half;
        dst[gq] = c4 < g.N ? *reinterpret_cast<const f32x4 *>(shrow + c4) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    };
    if constexpr (DN) {
      // Every load is issued before the first sum (cparts = 8 nv, nv <= 4).
      const int nv = g.cparts >> 3;
      f32x4 pv[MBW][4];
#pragma unroll
      for (int i = 0; i < MBW; ++i) {
        const int row = min(m0 + (wm * MBW + i) * 32 + r32, g.M - 1);
        const f32x4 *sp = reinterpret_cast<const f32x4 *>(g.css + (size_t)row * g.cparts) + half * nv;
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (v < nv) pv[i][v] = sp[v];
        mrow[i] = g.rowmod[row];
        if constexpr (kShAll) {
#pragma unroll
          for (int j = 0; j < TN; ++j) load_shift(i, j, shv[i][j]);
        }
      }
#pragma unroll
      for (int i = 0; i < MBW; ++i) {
        float ss = 0.f;
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (v < nv) ss = (((ss + pv[i][v][0]) + pv[i][v][1]) + pv[i][v][2]) + pv[i][v][3];
        ss += __shfl_xor(ss, 32, 64);
        rinv[i] = 1.0f / sqrtf(ss / (float)g.cd + g.ceps);
      }
    }
#pragma unroll
    for (int i = 0; i < MBW; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int rb = m0 + (wm * MBW + i) * 32, cb = n0 + (wn * TN + j) * 32;
        f32x4 sh1[4];
        if constexpr (DN && !kShAll) load_shift(i, j, sh1);
        // bf16 slot: 32 rows x 4 chunks of 16 B (8 bf16), chunk c of row r at
        // c ^ ((r / 4) % 4); this lane's 4 values are half `half` of chunk gq.
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
          float a0 = acc[i][j][4 * gq], a1 = acc[i][j][4 * gq + 1], a2 = acc[i][j][4 * gq + 2], a3 = acc[i][j][4 * gq + 3];
          if constexpr (DN) {
            const f32x4 sh = kShAll ? shv[kShAll ? i : 0][kShAll ? j : 0][gq] : sh1[gq];
            a0 = fmaf(a0, rinv[i], sh[0]);
            a1 = fmaf(a1, rinv[i], sh[1]);
            a2 = fmaf(a2, rinv[i], sh[2]);
            a3 = fmaf(a3, rinv[i], sh[3]);
          }
          if constexpr (EPI == kEpiGelu) {
            a0 = gelu_tanh_f(a0); a1 = gelu_tanh_f(a1); a2 = gelu_tanh_f(a2); a3 = gelu_tanh_f(a3);
          }
          bf16x4 o;
          o[0] = (bf16)a0; o[1] = (bf16)a1; o[2] = (bf16)a2; o[3] = (bf16)a3;
          const int c = gq ^ ((r32 >> 2) & 3);
          *reinterpret_cast<bf16x4 *>(stg + r32 * 64 + c * 16 + half * 8) = o;
        }
        // Pass p: rows 16 p + lane / 4, columns 8 (lane % 4) .. + 7.
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const int rr = 16 * p + (lane >> 2), c = lane & 3;
          const bf16x8 v = *reinterpret_cast<const bf16x8 *>(stg + rr * 64 + ((c ^ ((rr >> 2) & 3)) * 16));
          const int row = rb + rr, col = cb + c * 8;
          if (row < g.M && col < g.N) {
            const size_t off = g.out_rows > 0 ? kb32_offset(g.out_rows, row, col) : (size_t)row * g.ldo + col;
            *reinterpret_cast<bf16x8 *>(reinterpret_cast<bf16 *>(g.out) + off) = v;
          }
        }
      }
  }
}

template <typename T, int EPI, bool DN = false>
__global__ void __launch_bounds__(T::NT) gemm_bf16_kernel(GemmArgs g, int nrt, int nct, int ksplit) {
  constexpr int SBYTES = T::SBYTES;
  __shared__ __attribute__((aligned(1024))) uint8_t L[T::NST * SBYTES];

  // Work unit of this block: XCD x = b % 8 takes the x-th eighth of the unit
  // list; unit u is K slice u / n_tiles of tile u % n_tiles (one slice
  // unless the product is split).
  const int n_tiles = nrt * nct, n_units = n_tiles * ksplit;
  const int b = blockIdx.x, x = b & 7, q = b >> 3;
  const int per = n_units >> 3, extra = n_units & 7;
  if (q >= per + (x < extra ? 1 : 0)) return;
  const int unit = x * per + min(x, extra) + q;
  const int tile = unit % n_tiles, slice = unit / n_tiles;
  const int m0 = (tile / nct) * T::BM, n0 = (tile % nct) * T::BN;
  const int nks = g.K / T::BK / ksplit;
  f32x16 acc[T::MBW][T::TN];
  gemm_mainloop<T>(g, m0, n0, slice * nks, nks, L, acc);
  if constexpr (EPI == kEpiPartial) {
    GemmArgs gp = g;
    gp.out = g.part + (size_t)slice * g.M * g.N;
    gp.ldo = g.N;
    gemm_epilogue<T, EPI>(gp, m0, n0, L, acc);
  } else {
    gemm_epilogue<T, EPI, DN>(g, m0, n0, L, acc);
  }
}

// Block configurations and their measured cost on MI355X (one round of
// blocks over all CUs, microseconds): a per 1024 of K, plus b by epilogue
// (store, GELU, gated residual); least-squares fits to the projection shapes
// of the batch workloads at 1060, 2113, 4241 and 8482 rows (the 64-row tiles:
// at 50, 400, 800 and 1600 rows, where they can win).  Past K = 4096 a
// round costs a2 more per 1024 of K, from the 16384-deep MLP-down projection
// of a 26173-row VLM backbone batch (long sustained launches run each tile
// more slowly, by an amount that differs between tiles).
struct GemmCfg { int bm, bn, bk; float a, a2, b[3]; };
static constexpr GemmCfg kCfgs[kGemmConfigs] = {
    {384, 128, 32, 15.5f, 19.2f, {9.5f, 12.8f, 15.3f}},  // 0: 8 waves, 96 x 64 each
    {256, 256, 32, 18.8f, 13.8f, {9.2f, 12.3f, 16.7f}},  // 1: 16 waves, 64 x 64 each
    {128, 256, 32, 12.5f, 13.0f, {6.5f, 7.9f, 11.1f}},   // 2: 8 waves, 64 x 64 each
    {192, 128, 32, 10.7f, 3.2f, {4.9f, 5.5f, 9.4f}},     // 3: 8 waves, 96 x 32 each
    {288, 128, 32, 13.7f, 15.3f, {8.8f, 10.9f, 13.7f}},  // 4: 12 waves, 96 x 32 each
    {128, 64, 64, 4.7f, 5.0f, {3.1f, 3.4f, 6.0f}},       // 5: 4 waves, 64 x 32 each
    {192, 128, 64, 8.8f, 6.8f, {6.2f, 8.2f, 10.9f}},     // 6: 8 waves, 96 x 32 each
    {128, 128, 64, 6.5f, 6.0f, {4.7f, 6.3f, 9.9f}},      // 7: 4 waves, 64 x 64 each
    {160, 128, 64, 8.1f, 3.4f, {4.5f, 7.1f, 14.7f}},     // 8: 4 waves, 160 x 32 each
    {96, 128, 64, 5.5f, 4.2f, {4.3f, 6.0f, 8.9f}},       // 9: 4 waves, 96 x 32 each
    {256, 64, 64, 6.9f, 7.4f, {4.0f, 4.8f, 8.8f}},       // 10: 8 waves, 64 x 32 each
    {64, 64, 64, 2.8f, 5.0f, {4.2f, 4.1f, 6.8f}},        // 11: 4 waves, 32 x 32 each, 8 stages
    {64, 32, 64, 2.3f, 5.0f, {2.5f, 2.3f, 4.9f}},        // 12: 2 waves, 32 x 32 each, 8 stages
};
using Cfg0 = GemmTile<12, 2, 4, 2>;
using Cfg1 = GemmTile<8, 2, 4, 4>;
using Cfg2 = GemmTile<4, 2, 2, 4>;
using Cfg3 = GemmTile<6, 1, 2, 4>;
using Cfg4 = GemmTile<9, 1, 3, 4>;
using Cfg5 = GemmTile<4, 1, 2, 2, 64>;
using Cfg6 = GemmTile<6, 1, 2, 4, 64>;
using Cfg7 = GemmTile<4, 2, 2, 2, 64>;
using Cfg8 = GemmTile<5, 1, 1, 4, 64>;
using Cfg9 = GemmTile<3, 1, 1, 4, 64>;
using Cfg10 = GemmTile<8, 1, 4, 2, 64>;
using Cfg11 = GemmTile<2, 1, 2, 2, 64, 8>;
using Cfg12 = GemmTile<2, 1, 2, 1, 64, 8>;
template <typename T>
constexpr bool cfg_matches(const GemmCfg &c) { return T::BM == c.bm && T::BN == c.bn && T::BK == c.bk; }
static_assert(cfg_matches<Cfg0>(kCfgs[0]) && cfg_matches<Cfg1>(kCfgs[1]) && cfg_matches<Cfg2>(kCfgs[2]) &&
              cfg_matches<Cfg3>(kCfgs[3]) && cfg_matches<Cfg4>(kCfgs[4]) && cfg_matches<Cfg5>(kCfgs[5]) &&
              cfg_matches<Cfg6>(kCfgs[6]) && cfg_matches<Cfg7>(kCfgs[7]) && cfg_matches<Cfg8>(kCfgs[8]) &&
              cfg_matches<Cfg9>(kCfgs[9]) && cfg_matches<Cfg10>(kCfgs[10]) && cfg_matches<Cfg11>(kCfgs[11]) &&
              cfg_matches<Cfg12>(kCfgs[12]),
              "cost table matches the tiles");

// Sum of the K slices of a split product, in slice order, and the epilogue
// of the whole product; 4 consecutive columns per thread.
template <int EPI>
__global__ void __launch_bounds__(256) gemm_split_reduce_kernel(GemmArgs g, int ksplit) {
  const size_t n4 = (size_t)g.M * g.N / 4;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (size_t)gridDim.x * 256) {
    const size_t e = i * 4;
    const int row = (int)(e / g.N), col = (int)(e % g.N);
    f32x4 v = *reinterpret_cast<const f32x4 *>(g.part + e);
    for (int s2 = 1; s2 < ksplit; ++s2) {
      const f32x4 p = *reinterpret_cast<const f32x4 *>(g.part + (size_t)s2 * g.M * g.N + e);
      v[0] += p[0]; v[1] += p[1]; v[2] += p[2]; v[3] += p[3];
    }
    if constexpr (EPI == kEpiGatedResidual) {
      float *hp = reinterpret_cast<float *>(g.out) + (size_t)row * g.ldo + col;
      const float4 gt = *reinterpret_cast<const float4 *>(g.gate + (size_t)g.rowmod[row] * g.gate_stride + col);
      float4 hv = *reinterpret_cast<const float4 *>(hp);
      hv.x = hv.x + gt.x * v[0];
      hv.y = hv.y + gt.y * v[1];
      hv.z = hv.z + gt.z * v[2];
      hv.w = hv.w + gt.w * v[3];
      *reinterpret_cast<float4 *>(hp) = hv;
    } else {
      float a0 = v[0], a1 = v[1], a2 = v[2], a3 = v[3];
      if constexpr (EPI == kEpiGelu) {
        a0 = gelu_tanh_f(a0); a1 = gelu_tanh_f(a1); a2 = gelu_tanh_f(a2); a3 = gelu_tanh_f(a3);
      }
      bf16x4 o;
      o[0] = (bf16)a0; o[1] = (bf16)a1; o[2] = (bf16)a2; o[3] = (bf16)a3;
      const size_t off = g.out_rows > 0 ? kb32_offset(g.out_rows, row, col) : (size_t)row * g.ldo + col;
      *reinterpret_cast<bf16x4 *>(reinterpret_cast<bf16 *>(g.out) + off) = o;
    }
  }
}

// The same sum for a gated-residual product, fused with the modulated
// RMSNorm of the updated rows (the norm that reads them next).  One block per
// row, four columns per thread (N <= kFusedNormMax): sum the KS slices in
// slice order, apply the gated residual exactly as above, write the row back
// to h, and normalize it into u (row sum of squares: per wave, then the four
// wave sums in wave order), so a split product needs no separate norm launch.
template <int KS>
__global__ void __launch_bounds__(256) gemm_split_reduce_norm_kernel(GemmArgs g, NormArgs nm) {
  static_assert(kFusedNormMax == 4 * 256, "four columns per thread");
  __shared__ float wsum[4];
  const int row = blockIdx.x, i = threadIdx.x * 4;
  const int d = g.N;
  const size_t slice = (size_t)g.M * g.N;
  const int mod = g.rowmod[row];
  float *hr = reinterpret_cast<float *>(g.out) + (size_t)row * g.ldo;
  float4 hv = make_float4(0.f, 0.f, 0.f, 0.f);
  if (i < d) {
    const float *pr = g.part + (size_t)row * g.N + i;
    f32x4 p[KS];
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) p[s2] = *reinterpret_cast<const f32x4 *>(pr + s2 * slice);
    const float4 gt = *reinterpret_cast<const float4 *>(g.gate + (size_t)mod * g.gate_stride + i);
    hv = *reinterpret_cast<const float4 *>(hr + i);
    f32x4 a = p[0];
#pragma unroll
    for (int s2 = 1; s2 < KS; ++s2) { a[0] += p[s2][0]; a[1] += p[s2][1]; a[2] += p[s2][2]; a[3] += p[s2][3]; }
    hv.x = hv.x + gt.x * a[0];
    hv.y = hv.y + gt.y * a[1];
    hv.z = hv.z + gt.z * a[2];
    hv.w = hv.w + gt.w * a[3];
    *reinterpret_cast<float4 *>(hr + i) = hv;
  }
  const float ss = wave_sum(hv.x * hv.x + hv.y * hv.y + hv.z * hv.z + hv.w * hv.w);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float r = 1.0f / sqrtf((((wsum[0] + wsum[1]) + wsum[2]) + wsum[3]) / (float)d + nm.eps);
  if (i < d) {
    const float *mrow = nm.modtab + (size_t)mod * nm.mod_stride;
    const float4 a = *reinterpret_cast<const float4 *>(mrow + nm.scale_off + i);
    const float4 b = *reinterpret_cast<const float4 *>(mrow + nm.shift_off + i);
    bf16x4 o;
    o[0] = (bf16)(hv.x * r * (1.0f + a.x) + b.x);
    o[1] = (bf16)(hv.y * r * (1.0f + a.y) + b.y);
    o[2] = (bf16)(hv.z * r * (1.0f + a.z) + b.z);
    o[3] = (bf16)(hv.w * r * (1.0f + a.w) + b.w);
    const size_t off = nm.u_rows > 0 ? kb32_offset(nm.u_rows, row, i) : (size_t)row * d + i;
    *reinterpret_cast<bf16x4 *>(reinterpret_cast<bf16 *>(nm.u) + off) = o;
  }
}

// K slices for a launch of n_tiles tiles of BK-deep stages (1: no split).
// A product whose slice reduction also takes the norm that follows it
// (fused) costs no extra launch, so it splits up to a whole round of blocks
// (kSplitMinTilesNorm tiles); others only below kSplitMinTiles.
int gemm_split_count(const GemmArgs &g, int n_tiles, int bk, bool fused) {
  // K = 1024 products are too short for the saving to pay for the second launch.
  if (!g.part || n_tiles >= (fused ? kSplitMinTilesNorm : kSplitMinTiles) || g.K < 2048 || g.N % 4 || g.ldo % 4)
    return 1;
  const int nk = g.K / bk;
  const int most_blocks = fused ? std::max(256, 2 * kSplitMinTilesNorm) : 256;
  for (int ks = kSplitMax; ks >= 2; ks /= 2)
    if (n_tiles * ks <= most_blocks && nk % ks == 0 && nk / ks >= 4 && (size_t)ks * g.M * g.N <= g.part_floats)
      return ks;
  return 1;
}

// Whether a split gated-residual product can take the norm that follows it.
static bool fusable_norm(const GemmArgs &g, const NormArgs *nm) {
  return nm && nm->u && g.epi == kEpiGatedResidual && g.N <= kFusedNormMax && g.N % 4 == 0 && g.ldo % 4 == 0 &&
         (nm->u_rows == 0 || (nm->u_rows >= g.M && g.N % 32 == 0));
}

template <typename T>
static hipError_t launch_tile(const GemmArgs &g, hipStream_t s, bool allow_split, const NormArgs *nm,
                              bool *normed, bool *deferred) {
  const int nrt = (g.M + T::BM - 1) / T::BM, nct = (g.N + T::BN - 1) / T::BN;
  // A launch that completes a deferred norm is never split.
  const bool completes = g.css && (g.epi == kEpiStore || g.epi == kEpiGelu);
  const int ks = allow_split && !completes ? gemm_split_count(g, nrt * nct, T::BK, fusable_norm(g, nm)) : 1;
  dim3 grid((nrt * nct * ks + 7) / 8 * 8);
  if (ks > 1) {
    hipLaunchKernelGGL((gemm_bf16_kernel<T, kEpiPartial>), grid, dim3(T::NT), 0, s, g, nrt, nct, ks);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (fusable_norm(g, nm)) {
      const dim3 ngrid(g.M);
      switch (ks) {
        case 2: hipLaunchKernelGGL(gemm_split_reduce_norm_kernel<2>, ngrid, dim3(256), 0, s, g, *nm); break;
        case 4: hipLaunchKernelGGL(gemm_split_reduce_norm_kernel<4>, ngrid, dim3(256), 0, s, g, *nm); break;
        default: hipLaunchKernelGGL(gemm_split_reduce_norm_kernel<kSplitMax>, ngrid, dim3(256), 0, s, g, *nm); break;
      }
      if (normed) *normed = true;
      return hipGetLastError();
    }
    const int rgrid = (int)std::min<size_t>(((size_t)g.M * g.N / 4 + 255) / 256, 4096);
    switch (g.epi) {
      case kEpiStore: hipLaunchKernelGGL(gemm_split_reduce_kernel<kEpiStore>, dim3(rgrid), dim3(256), 0, s, g, ks); break;
      case kEpiGelu: hipLaunchKernelGGL(gemm_split_reduce_kernel<kEpiGelu>, dim3(rgrid), dim3(256), 0, s, g, ks); break;
      default: hipLaunchKernelGGL(gemm_split_reduce_kernel<kEpiGatedResidual>, dim3(rgrid), dim3(256), 0, s, g, ks); break;
    }
    return hipGetLastError();
  }
  if (g.dt && g.epi == kEpiGatedResidual) {
    hipLaunchKernelGGL((gemm_bf16_kernel<T, kEpiGatedResidual, true>), grid, dim3(T::NT), 0, s, g, nrt, nct, 1);
    if (deferred) *deferred = true;
    return hipGetLastError();
  }
  if (completes) {
    if (g.epi == kEpiGelu) hipLaunchKernelGGL((gemm_bf16_kernel<T, kEpiGelu, true>), grid, dim3(T::NT), 0, s, g, nrt, nct, 1);
    else hipLaunchKernelGGL((gemm_bf16_kernel<T, kEpiStore, true>), grid, dim3(T::NT), 0, s, g, nrt, nct, 1);
    return hipGetLastError();
  }
  switch (g.epi) {
    case kEpiStore: hipLaunchKernelGGL((gemm_bf16_kernel<T, kEpiStore>), grid, dim3(T::NT), 0, s, g, nrt, nct, 1); break;
    case kEpiGelu: hipLaunchKernelGGL((gemm_bf16_kernel<T, kEpiGelu>), grid, dim3(T::NT), 0, s, g, nrt, nct, 1); break;
    default: hipLaunchKernelGGL((gemm_bf16_kernel<T, kEpiGatedResidual>), grid, dim3(T::NT), 0, s, g, nrt, nct, 1); break;
  }
  return hipGetLastError();
}

static hipError_t launch_cfg(const GemmArgs &g, int cfg, hipStream_t s, bool allow_split,
                             const NormArgs *nm = nullptr, bool *normed = nullptr, bool *deferred = nullptr) {
  if (g.M <= 0) return hipSuccess;
  if (g.K % 128 != 0 || g.N % 8 != 0 || g.a_rows < g.M) return hipErrorInvalidValue;
  switch (cfg) {
    case 0: return launch_tile<Cfg0>(g, s, allow_split, nm, normed, deferred);
    case 1: return launch_tile<Cfg1>(g, s, allow_split, nm, normed, deferred);
    case 2: return launch_tile<Cfg2>(g, s, allow_split, nm, normed, deferred);
    case 3: return launch_tile<Cfg3>(g, s, allow_split, nm, normed, deferred);
    case 4: return launch_tile<Cfg4>(g, s, allow_split, nm, normed, deferred);
    case 5: return launch_tile<Cfg5>(g, s, allow_split, nm, normed, deferred);
    case 6: return launch_tile<Cfg6>(g, s, allow_split, nm, normed, deferred);
    case 7: return launch_tile<Cfg7>(g, s, allow_split, nm, normed, deferred);
    case 8: return launch_tile<Cfg8>(g, s, allow_split, nm, normed, deferred);
    case 9: return launch_tile<Cfg9>(g, s, allow_split, nm, normed, deferred);
    case 10: return launch_tile<Cfg10>(g, s, allow_split, nm, normed, deferred);
    case 11: return launch_tile<Cfg11>(g, s, allow_split, nm, normed, deferred);
    case 12: return launch_tile<Cfg12>(g, s, allow_split, nm, normed, deferred);
    default: return hipErrorInvalidValue;
  }
}

static int device_cu_count();

// Whether launch_gemm(g, true, s, force_cfg, then_norm) with g.dt set takes
// the deferred norm (an unsplit gated-residual launch) for these sizes.
bool gemm_defers(const GemmArgs &g, int force_cfg, const NormArgs *then_norm) {
  if (g.M <= 0 || g.epi != kEpiGatedResidual) return false;
  if (force_cfg >= 0) return true;
  const int c = gemm_pick_config(g.M, g.N, g.K, g.epi, device_cu_count());
  const int n_tiles = ((g.M + kCfgs[c].bm - 1) / kCfgs[c].bm) * ((g.N + kCfgs[c].bn - 1) / kCfgs[c].bn);
  return gemm_split_count(g, n_tiles, kCfgs[c].bk, fusable_norm(g, then_norm)) == 1;
}

// Shift halves of deferred norms: one thread per output column of one layer's
// product, for up to kShiftRows modulation rows at a time; the rows' shift
// vectors pass through LDS kShiftK values of K at a time (K-major, so one
// 16-byte read serves four rows).  Column n of a kb32 weight holds its K
// values in 64-byte runs, one per 32 of K.
constexpr int kShiftRows = 16, kShiftK = 256;
__global__ void __launch_bounds__(256) shift_proj_kernel(const float *__restrict__ modtab, int mod_stride, int n_mod,
                                                         int layer_stride, int q_off, int u_off, int d,
                                                         const bf16 *__restrict__ wq, int Nq,
                                                         const bf16 *__restrict__ wu, int Nu, int nbq,
                                                         float *__restrict__ S) {
  __shared__ __attribute__((aligned(16))) float sh[kShiftK][kShiftRows];
  const int l = blockIdx.y, r0 = blockIdx.z * kShiftRows, nr = min(kShiftRows, n_mod - r0);
  const bool isq = (int)blockIdx.x < nbq;
  const int col = (isq ? (int)blockIdx.x : (int)blockIdx.x - nbq) * 256 + threadIdx.x;
  const int N = isq ? Nq : Nu, off = isq ? q_off : u_off;
  const bf16 *W = (isq ? wq : wu) + (size_t)l * N * d;
  float acc[kShiftRows];
#pragma unroll
  for (int r = 0; r < kShiftRows; ++r) acc[r] = 0.f;
  for (int k0 = 0; k0 < d; k0 += kShiftK) {
    const int kn = min(kShiftK, d - k0);
    __syncthreads();                        // the previous chunk's reads are done
    for (int i = threadIdx.x; i < kShiftK * kShiftRows; i += 256) {
      const int k = i / kShiftRows, r = i % kShiftRows;
      sh[k][r] = (r < nr && k < kn) ? modtab[(size_t)(r0 + r) * mod_stride + (size_t)l * layer_stride + off + k0 + k]
                                    : 0.f;
    }
    __syncthreads();
    if (col < N) {
      for (int kb = 0; kb < kn; kb += 32) {
        const bf16 *wp = W + ((size_t)((k0 + kb) >> 5) * N + col) * 32;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const bf16x8 w8 = *reinterpret_cast<const bf16x8 *>(wp + 8 * c);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float w = (float)w8[e];
            const float4 *sv = reinterpret_cast<const float4 *>(&sh[kb + 8 * c + e][0]);
#pragma unroll
            for (int r4 = 0; r4 < kShiftRows / 4; ++r4) {
              const float4 v = sv[r4];
              acc[4 * r4] = fmaf(v.x, w, acc[4 * r4]);
              acc[4 * r4 + 1] = fmaf(v.y, w, acc[4 * r4 + 1]);
              acc[4 * r4 + 2] = fmaf(v.z, w, acc[4 * r4 + 2]);
              acc[4 * r4 + 3] = fmaf(v.w, w, acc[4 * r4 + 3]);
            }
          }
        }
      }
    }
  }
  if (col < N) {
    const int Nt = Nq + Nu;
#pragma unroll
    for (int r = 0; r < kShiftRows; ++r)
      if (r < nr) S[((size_t)l * n_mod + r0 + r) * Nt + (isq ? 0 : Nq) + col] = acc[r];
  }
}

hipError_t launch_shift_proj(const float *modtab, int mod_stride, int n_mod, int L, int layer_stride, int q_off,
                             int u_off, int d, const void *wq, int Nq, const void *wu, int Nu, float *S,
                             hipStream_t s) {
  if (n_mod <= 0 || L <= 0) return hipSuccess;
  if (d % 32 != 0 || Nq <= 0 || Nu <= 0) return hipErrorInvalidValue;
  const int nbq = (Nq + 255) / 256, nbu = (Nu + 255) / 256;
  const dim3 grid(nbq + nbu, L, (n_mod + kShiftRows - 1) / kShiftRows);
  hipLaunchKernelGGL(shift_proj_kernel, grid, dim3(256), 0, s, modtab, mod_stride, n_mod, layer_stride, q_off, u_off,
                     d, reinterpret_cast<const bf16 *>(wq), Nq, reinterpret_cast<const bf16 *>(wu), Nu, nbq, S);
  return hipGetLastError();
}

// A forced configuration never splits K: every configuration then computes
// each output with the same instruction sequence.
hipError_t launch_gemm_cfg(const GemmArgs &g, int cfg, hipStream_t s) { return launch_cfg(g, cfg, s, false); }

int gemm_pick_config(int M, int N, int K, int epi, int n_cu) {
  const int e = epi < 0 || epi > 2 ? 2 : epi;
  int best = 0;
  float best_t = 0.f;
  for (int c = 0; c < kGemmConfigs; ++c) {
    const long tiles = (long)((M + kCfgs[c].bm - 1) / kCfgs[c].bm) * ((N + kCfgs[c].bn - 1) / kCfgs[c].bn);
    const long rounds = (tiles + n_cu - 1) / n_cu;
    const float t = rounds * (kCfgs[c].a * (K / 1024.0f) + kCfgs[c].a2 * (std::max(K - 4096, 0) / 1024.0f) +
                              kCfgs[c].b[e]);
    if (best_t == 0.f || t < best_t) { best = c; best_t = t; }
  }
  return best;
}

template <int EPI>
__device__ __forceinline__ void epilogue_f32(const GemmArgs &g, int row, int col, float v) {
  float *out = reinterpret_cast<float *>(g.out) + (size_t)row * g.ldo + col;
  if constexpr (EPI == kEpiStore) *out = v;
  else if constexpr (EPI == kEpiGelu) *out = gelu_tanh_f(v);
  else *out = *out + g.gate[(size_t)g.rowmod[row] * g.gate_stride + col] * v;
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
      if (col < g.N) epilogue_f32<EPI>(g, row, col, acc[i][j]);
    }
  }
}

// Compute units of the current device, cached per device (any host thread).
static int device_cu_count() {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> cache[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v > 0) return v;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
  cache[dev].store(v, std::memory_order_relaxed);
  return v;
}

hipError_t launch_gemm(const GemmArgs &g, bool bf16_mode, hipStream_t s, int force_cfg, const NormArgs *then_norm,
                       bool *normed, bool *deferred) {
  if (normed) *normed = false;
  if (deferred) *deferred = false;
  if (g.M <= 0) return hipSuccess;
  if (bf16_mode) {
    const int n_cu = device_cu_count();
    if ((g.dt || g.css) && (g.N % 32 != 0 || (g.css && (g.cparts <= 0 || g.cparts % 8 || g.cparts > 32 || g.cd <= 0))))
      return hipErrorInvalidValue;
    if (force_cfg >= 0) return launch_cfg(g, force_cfg, s, false, nullptr, nullptr, deferred);
    return launch_cfg(g, gemm_pick_config(g.M, g.N, g.K, g.epi, n_cu), s, true, then_norm, normed, deferred);
  }
  if (g.dt || g.css) return hipErrorInvalidValue;   // bf16 only
  dim3 grid((g.N + 63) / 64, (g.M + 63) / 64);
  switch (g.epi) {
    case kEpiStore: hipLaunchKernelGGL(gemm_f32_kernel<kEpiStore>, grid, dim3(256), 0, s, g); break;
    case kEpiGelu: hipLaunchKernelGGL(gemm_f32_kernel<kEpiGelu>, grid, dim3(256), 0, s, g); break;
    default: hipLaunchKernelGGL(gemm_f32_kernel<kEpiGatedResidual>, grid, dim3(256), 0, s, g); break;
  }
  return hipGetLastError();
}

}  // namespace rosa
