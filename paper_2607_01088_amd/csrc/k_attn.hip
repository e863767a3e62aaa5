// Ragged prefix + action attention of one layer.
//
// Request r's H_r action tokens (G = n_q / n_kv query heads per KV head, so
// G*H_r query rows per KV head) attend to its own key sequence: the P_r cached
// prefix keys of this layer followed by its H_r action keys; no other request
// and no padding is visible.  Scale 1/sqrt(head_dim); no causal mask.
//
// bf16 kernel (gfx950 MFMA).  A work item is (request, KV head, up to 128 NG
// query rows, key range).  Its four waves stream the key range through LDS in
// 32-key tiles: a K ring of three stages and a V ring of two, filled by
// global_load_lds_dwordx4 (step t issues V tile t + 1 and K tile t + 2).
// Each wave owns NG groups of 32 query rows (groups w and w + 4 of the item),
// so every K and V fragment it reads from LDS feeds the MFMAs of all its
// groups; NG is 2 where Q^T and O^T of two groups fit the register file
// (head_dim <= 64) and 1 otherwise.  Step t computes S^T = K Q^T of tile t
// with v_mfma_f32_32x32x16_bf16 (K from LDS, Q^T held in registers for the
// whole item; each lane owns one query column, so softmax statistics are
// in-lane), its softmax, and O^T += V^T P^T (P^T from registers, V^T from
// the row-major V tile through the LDS transpose read ds_read_b64_tr_b16).
// Every MFMA's LDS operand is read two fragments ahead.  The softmax uses a fixed reference
// max per query (its first tile's), so the output accumulators are never
// rescaled; a block whose later scores overshoot that reference runs again
// with the true max.  Work items that cover part of a request's keys write
// unnormalized partial results that a merge kernel combines in a fixed order.
#include <math.h>

#include <type_traits>

#include "rosa_device.h"
#include "rosa_internal.h"

namespace rosa {

namespace at {
constexpr int TK = 32;   // keys per LDS stage
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
constexpr int waitcnt_lgkm0 = 15 | (3 << 14) | (7 << 4);   // lgkmcnt(0), others unconstrained
// Chunk swizzle of LDS rows: 16-byte chunk c of row r is stored at c ^ swz(r),
// swz(r) = the two 2-bit halves of r % 16 swapped.  The 16 consecutive rows
// that one 16-lane group reads at one chunk (K operand), and the 4 rows x 4
// chunks that the transpose reads of a 32-lane half touch (V operand), then
// fall in distinct bank groups.
__device__ __forceinline__ int swz(int r, int cpr) { return (((r & 3) << 2) | ((r >> 2) & 3)) & (cpr - 1); }
}  // namespace at



typedef __attribute__((address_space(3))) const uint8_t lds_u8;
__device__ __forceinline__ const lds_u8 *lds_ptr(uint32_t a) { return (const lds_u8 *)(size_t)a; }
__device__ __forceinline__ bf16x8 lds_tr_pair(const lds_u8 *p0, const lds_u8 *p1) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  const i16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(p0));
  const i16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(p1));
  const uint2 u0 = __builtin_bit_cast(uint2, v0);
  const uint2 u1 = __builtin_bit_cast(uint2, v1);
  return __builtin_bit_cast(bf16x8, make_uint4(u0.x, u0.y, u1.x, u1.y));
}
template <int HD, int NG>
struct AttnTile {
  static constexpr int ROWB = HD * 2;             // bytes per K or V row
  static constexpr int CPR = ROWB / 16;           // 16-byte chunks per row
  static constexpr int TILEB = 32 * ROWB;         // bytes of one 32-key K (or V) tile
  static constexpr int UNITS = TILEB / 1024;      // 1 KB copies per tile
  static constexpr int UPW = (UNITS + 3) / 4;     // copies per copying wave per tile
  static constexpr int RPU = 1024 / ROWB;         // rows per 1 KB copy
  static constexpr int KST = 3, VST = 2;          // K ring and V ring depths
  static constexpr int RINGB = (KST + VST) * TILEB;
  static constexpr int STGB = 4 * NG * 32 * 2 * HD;   // output staging of the block's query rows
  static constexpr int LDSB = RINGB > STGB ? RINGB : STGB;
  static_assert(UNITS % 4 == 0 || UNITS < 4, "copy split");
};

// Two blocks of four waves share a CU (two waves per SIMD): the register file
// (at most 256 per lane) and LDS (at most 80 KB) are sized for that, and each
// SIMD interleaves the two waves, so one wave's LDS waits and softmax work
// overlap the other's MFMAs.  A wave owns NG groups of 32 query rows (groups
// w and w + 4 of the item).  Step t (one 32-key tile): wait for K tile t and
// V tile t, one barrier, issue the copies of V tile t + 1 and K tile t + 2,
// S^T = K Q^T, the softmax of the tile, O^T += V^T P^T.
// CAUSAL: the prefix producer's launches with causal segments; each query
// row additionally masks the keys at or past its token's limit
// max(causal_b, t + 1) in the tiles that reach it.
template <int HD, int NG, bool CAUSAL>
__global__ void __launch_bounds__(256, 2) attention_bf16_kernel(AttnArgs a) {
  using at::TK;
  using T = AttnTile<HD, NG>;
  constexpr int NS = HD / 16;       // MFMA k-steps over head_dim for S
  constexpr int NT = HD / 32;       // 32-row output tiles over head_dim
  constexpr int CPR = T::CPR, ROWB = T::ROWB, TILEB = T::TILEB, UPW = T::UPW;
  constexpr int KST = T::KST, VST = T::VST;
  // K stage s at s TILEB (s < 3), V stage s at (3 + s) TILEB (s < 2).  Every
  // stage offset from a lane base fits a ds_read immediate.
  __shared__ __attribute__((aligned(1024))) uint8_t smem[T::LDSB];
  static_assert(T::RINGB <= 65536 + TILEB, "stage offsets must fit the LDS immediate");

  // The block is persistent: it runs the items of its list (a.ordered[b],
  // then each entry's `next`) one after another.
  if (a.ordered[blockIdx.x].nq <= 0) return;
  const int G = a.nq / a.nkv;
  const bf16 *qkv = reinterpret_cast<const bf16 *>(a.qkv);
  const size_t prow = (size_t)a.nkv * HD;   // prefix row stride (elements)
  const long ldq = a.ldqkv;
  const uint32_t lds0 = lds_u32(smem);

  for (int e = blockIdx.x; e >= 0;) {
  // The item's words pass through readfirstlane: the kernel's own stores
  // keep the compiler from proving the table unchanged (so from loading it
  // with scalar loads), and every field must be wave-uniform.
  AttnItem it;
  {
    static_assert(sizeof(AttnItem) % 4 == 0, "item is whole words");
    const uint32_t *src = reinterpret_cast<const uint32_t *>(a.ordered + e);
    uint32_t w[sizeof(AttnItem) / 4];
#pragma unroll
    for (int i = 0; i < (int)(sizeof(AttnItem) / 4); ++i) w[i] = __builtin_amdgcn_readfirstlane(src[i]);
    __builtin_memcpy(&it, w, sizeof(AttnItem));
  }
  e = it.next;
  // The thread index is taken through an opaque copy per item, so the
  // compiler does not hoist the per-lane addresses derived from it out of the
  // item loop (they would hold registers across every item).
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & 3;   // wave-uniform, in an SGPR
  const int half = lane >> 5;
  const bf16 *pk = reinterpret_cast<const bf16 *>(it.pk) + (size_t)a.layer * it.P * prow + (size_t)it.kvh * HD;
  const bf16 *pv = reinterpret_cast<const bf16 *>(it.pv) + (size_t)a.layer * it.P * prow + (size_t)it.kvh * HD;
  const bf16 *ak = qkv + (size_t)it.tok_off * a.ldqkv + (size_t)(a.nq + it.kvh) * HD;
  const bf16 *av = qkv + (size_t)it.tok_off * a.ldqkv + (size_t)(a.nq + a.nkv + it.kvh) * HD;
  // Tile t covers keys [k0 + 32 t, k0 + 32 t + 32) with k0 = kend - 32 nkt:
  // only tile 0 can reach below kbeg (those keys are masked), so the key
  // loop itself never masks.
  const int nkt = (it.kend - it.kbeg + TK - 1) / TK;
  const int k0 = it.kend - TK * nkt;

  // Copies: 1 KB units, unit u of a tile by wave u % 4; lane i fills physical
  // chunk i % CPR of row u * RPU + i / CPR, which holds logical chunk
  // (i % CPR) ^ swz(row).  A tile wholly in the prefix takes its sources from
  // a wave-uniform base plus per-lane byte offsets fixed for the whole item;
  // the others (at most two per item) compute each lane's key: keys below the
  // range load the first valid key (finite values; their scores are masked).
  // Tile indices past the last tile copy the last tile again into a stage no
  // step reads, so every step issues the same number of copies.
  uint32_t poff[UPW];
#pragma unroll
  for (int j = 0; j < UPW; ++j) {
    const int row = (4 * j + wave) * T::RPU + lane / CPR;
    poff[j] = (uint32_t)((row * (int)prow + (((lane % CPR) ^ at::swz(row, CPR)) << 3)) * 2);
  }
  auto copy_tile = [&](int t, const bf16 *pbase, const bf16 *abase, uint32_t dst_stage) __attribute__((always_inline)) {
    const int kt0 = k0 + max(0, min(t, nkt - 1)) * TK;
    if (kt0 >= it.kbeg && kt0 + TK <= it.P) {
      const bf16 *b = pbase + (size_t)kt0 * prow;
#pragma unroll
      for (int j = 0; j < UPW; ++j)
        if (4 * j + wave < T::UNITS) dma_1k_s(b, poff[j], dst_stage + (4 * j + wave) * 1024);
    } else {
      // Recomputed from an opaque copy of the lane index at every use, so the
      // compiler does not hoist these per-lane addresses out of the key loop
      // (they would hold registers for the whole item).
      int ln = lane;
      asm volatile("" : "+v"(ln));
#pragma unroll
      for (int j = 0; j < UPW; ++j) {
        if (4 * j + wave >= T::UNITS) continue;
        const int row = (4 * j + wave) * T::RPU + ln / CPR;
        const int c = (ln % CPR) ^ at::swz(row, CPR);
        const int key = max(kt0 + row, it.kbeg);
        const bool pre = key < it.P;
        const long roff = (pre ? (long)key * (long)prow : (long)(key - it.P) * ldq) + c * 8;
        dma_1k((pre ? pbase : abase) + roff, dst_stage + (4 * j + wave) * 1024);
      }
    }
  };
  auto kstage = [&](int s) { return lds0 + (uint32_t)(s * TILEB); };
  auto vstage = [&](int s) { return lds0 + (uint32_t)((KST + s) * TILEB); };

  // K operand: row lane%32, logical chunk 2 ks + half at physical chunk
  // (2 ks + half) ^ swz(row).  The swizzle's upper bits act on bits 5.. of
  // the byte offset, which the row offset (a multiple of ROWB >= 64) and the
  // 1 KB-aligned ring leave clear, so the address of k-step ks < 8 is one
  // base XOR 32 ks; k-steps 8 apart differ by 256 bytes (an immediate).
  const int krow = lane & 31;
  uint32_t kbase;
  {
    const int sw = at::swz(krow, CPR);
    kbase = (lds0 + krow * ROWB + ((half ^ (sw & 1)) << 4)) ^ ((uint32_t)(sw >> 1) << 5);
  }
  // V transpose reads: source lane s of 16-lane group G16 reads 8 bytes at
  // row 16 ks + 4 half + s/4 (and 8 rows further), head-dim column
  // 32 n + 16 G16 + 4 (s%4).  Output tile n < 4 sits at base XOR 64 n (the
  // swizzle's upper bits act on bits 6-7 only); tiles 4 apart differ by 256
  // bytes, k-steps by 16 rows.
  const int src16 = lane & 15, g16 = (lane >> 4) & 1;
  uint32_t vbase[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int r = half * 4 + (src16 >> 2) + 8 * h;
    const int sw = at::swz(r, CPR);
    const int cl = (2 * g16 + ((src16 >> 1) & 1)) ^ (sw & 3);
    vbase[h] = (lds0 + KST * TILEB + r * ROWB + 16 * cl + 8 * (src16 & 1)) ^ ((uint32_t)(sw >> 2) << 6);
  }
  auto kfrag = [&](int kst, int i) __attribute__((always_inline)) -> bf16x8 {
    return *reinterpret_cast<const __attribute__((address_space(3))) bf16x8 *>(
        lds_ptr(kbase ^ (uint32_t)(32 * (i % 8))) + kst * TILEB + (i / 8) * 256);
  };
  auto vfrag = [&](int vst, int j) __attribute__((always_inline)) -> bf16x8 {
    const int ks = j / NT, n = j % NT;
    const int c = vst * TILEB + (n / 4) * 256 + ks * 16 * ROWB;
    const uint32_t x = (uint32_t)(64 * (n % 4));
    return lds_tr_pair(lds_ptr(vbase[0] ^ x) + c, lds_ptr(vbase[1] ^ x) + c);
  };

  // Q^T operand of group g, held for the whole item: lane holds
  // Q[row][16 s + 8 half .. + 7] for its row; rows past the item's queries
  // read the item's first row instead (their results are never stored).
  bf16x8 qf[NG][NS];
  auto load_q = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const int loc = 32 * (wave + 4 * g) + (lane & 31);
      const int qrow = it.q0 + (loc < it.nq ? loc : 0);
      const bf16 *qp = qkv + (size_t)(it.tok_off + qrow / G) * a.ldqkv + (size_t)(it.kvh * G + qrow % G) * HD + half * 8;
#pragma unroll
      for (int s = 0; s < NS; ++s) qf[g][s] = *reinterpret_cast<const bf16x8 *>(qp + 16 * s);
    }
  };

  f32x16 o[NG][NT];
  // Softmax without rescaling the output inside the key loop: each query's
  // reference max m_ref is its max over the item's first 32-key tile, and
  // P = 2^((s - m_ref) log2(e) / sqrt(hd)) may exceed 1.  If a tile's sum of P
  // exceeds 2^64 (room to spare below fp32 overflow for the running sums),
  // the block finds every query's true max and runs the item again with it as
  // reference, where P <= 1.  Either way the output accumulators are only
  // touched by MFMAs in the loop.  The two 32-lane halves hold different keys
  // of the same query: they keep their own sums, combined at the end.
  float m_ref[NG], m_true[NG], l_run[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) m_true[g] = -INFINITY;
  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);   // log2(e) / sqrt(hd)
  int ovf = 0;

  // S^T (32 keys x 32 queries; lane = query lane%32, register r = key
  // (r/4)*8 + 4 half + r%4) of K stage kst for every group.  Each slot (one
  // scheduling region) issues the read of fragment i + 2 and the MFMAs of
  // fragment i, so reads run two ahead and no more fragments are held in
  // registers (the same holds for the V^T fragments of O^T += V^T P^T).
  auto scores = [&](int kst, f32x16 (&s)[NG]) __attribute__((always_inline)) {
    bf16x8 fr[3];
    fr[0] = kfrag(kst, 0);
    fr[1] = kfrag(kst, 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      if (i + 2 < NS) fr[(i + 2) % 3] = kfrag(kst, i + 2);
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        // the first k-step accumulates onto an inline zero (no register clearing)
        const f32x16 c = i == 0 ? f32x16{} : s[g];
        s[g] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[i % 3], qf[g][i], c, 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // O^T += V^T P^T over V stage vst: P^T k-step ks is registers 8 ks .. 8 ks + 7
  // of the score tile (keys permuted identically on both operands).
  auto pv_acc = [&](int vst, const bf16x8 (&pp)[NG][2]) __attribute__((always_inline)) {
    constexpr int NJ = 2 * NT;
    bf16x8 fr[3];
    fr[0] = vfrag(vst, 0);
    fr[1] = vfrag(vst, 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      if (j + 2 < NJ) fr[(j + 2) % 3] = vfrag(vst, j + 2);
      const int ks = j / NT, n = j % NT;
#pragma unroll
      for (int g = 0; g < NG; ++g) o[g][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[j % 3], pp[g][ks], o[g][n], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // Causal limits: key j is visible to this lane's query row of group g iff
  // j < lim(g) (rows past the item's queries never mask).  Only the wave's
  // smallest limit, lim_lo (wave-uniform), is held through the key loop: it
  // tells the tiles that need the mask, which recomputes the lane's limits.
  auto causal_lim = [&](int g, int ln) __attribute__((always_inline)) -> int {
    const int loc = 32 * (wave + 4 * g) + (ln & 31);
    return loc < it.nq ? max(it.causal_b, (it.q0 + loc) / G + 1) : 0x7fffffff;
  };
  int lim_lo = 0x7fffffff;
  if constexpr (CAUSAL) {
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      int v = causal_lim(g, lane);
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
      lim_lo = min(lim_lo, __builtin_amdgcn_readfirstlane(v));
    }
  }
  auto mask_causal = [&](f32x16 (&s)[NG], int kt0) __attribute__((always_inline)) {
    int ln = lane;
    asm volatile("" : "+v"(ln));            // recomputed here, not held through the loop
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const int lim = causal_lim(g, ln);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kt0 + (r >> 2) * 8 + ((ln >> 5) & 1) * 4 + (r & 3);
        if (key >= lim) s[g][r] = -INFINITY;
      }
    }
  };
  // Keys of the item's first tile below its key range take no weight.
  auto mask_first = [&](f32x16 (&s)[NG]) __attribute__((always_inline)) {
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + (r >> 2) * 8 + half * 4 + (r & 3);
        if (key < it.kbeg) s[g][r] = -INFINITY;
      }
  };
  auto tile_max = [&](const f32x16 &s) __attribute__((always_inline)) -> float {
    float tmax = fmaxf(s[0], s[1]);
#pragma unroll
    for (int r = 2; r < 16; ++r) tmax = fmaxf(tmax, s[r]);
    return tmax;
  };
  // Softmax of one tile into P^T (bf16) and its sum.  The sum is taken over
  // the bf16 values that enter O += V^T P^T (two per dot-product instruction),
  // so numerator and denominator see the same weights.  A sum above 2^64 (or
  // not finite) means a score overshot the reference by about that much: the
  // block then finds the true maxima and runs the item again.
  auto softmax = [&](f32x16 (&s)[NG], bf16x8 (&pp)[NG][2]) __attribute__((always_inline)) {
    typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
    const bf16x2 ones = {(bf16)1.0f, (bf16)1.0f};
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const float mb = -m_ref[g] * sl2;
#pragma unroll
      for (int r = 0; r < 16; ++r) s[g][r] = __builtin_amdgcn_exp2f(fmaf(s[g][r], sl2, mb));
      // Pairs are packed one at a time and P^T is assembled from the packed
      // words (extracting words from a packed bf16 vector was mis-lowered).
      float ps = 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          bf16x2 p2;
          p2[0] = (bf16)s[g][8 * h + 2 * e];
          p2[1] = (bf16)s[g][8 * h + 2 * e + 1];
          ps = __builtin_amdgcn_fdot2_f32_bf16(p2, ones, ps, false);
          w[e] = __builtin_bit_cast(uint32_t, p2);
        }
        pp[g][h] = __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
      }
      ovf |= !(ps <= 0x1p64f);
      l_run[g] += ps;
    }
  };

  // vmcnt after which this wave's copies of K tile t and V tile t have landed
  // at step t: the K copies of tile t + 1 (issued last) may still be in flight.
  constexpr int WAIT = at::waitcnt_vm(UPW);
  // Step t with K tile t in K stage KS = t % 3 and V tile t in V stage VS =
  // t % 2 (compile-time, so every stage offset is an immediate): wait for
  // both, refill the stages tile t - 1 left with V tile t + 1 and K tile
  // t + 2, then S, softmax and O += P V.  The LDS bases are re-pinned per step
  // so the compiler keeps one register per base rather than hoisting every
  // derived address out of the loop.
  //   MODE 0: softmax against m_ref and O += P V; on the first tile (t == 0)
  //           the keys below the range are masked and, if set_ref, m_ref is
  //           set to the first tile's maxima.
  //   MODE 1: the maxima only (m_true), for a block whose first pass overflowed.
  auto step = [&](int t, auto ks_t, auto vs_t, auto mode_t, bool set_ref) __attribute__((always_inline)) {
    constexpr int KS = decltype(ks_t)::value, VS = decltype(vs_t)::value, MODE = decltype(mode_t)::value;
    __builtin_amdgcn_s_waitcnt(WAIT);       // this wave's copies of K tile t and V tile t have landed
    __builtin_amdgcn_s_barrier();           // ... and every wave's; the stages of tile t - 1 are free
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" : "+v"(kbase), "+v"(vbase[0]), "+v"(vbase[1]));
    copy_tile(t + 1, pv, av, vstage(VS ^ 1));
    copy_tile(t + 2, pk, ak, kstage((KS + 2) % 3));
    __builtin_amdgcn_sched_barrier(0);
    f32x16 sc[NG];
    scores(KS, sc);
    if (t == 0) mask_first(sc);
    if constexpr (CAUSAL) {
      if (k0 + TK * t + TK > lim_lo) mask_causal(sc, k0 + TK * t);
    }
    if constexpr (MODE == 1) {
#pragma unroll
      for (int g = 0; g < NG; ++g) m_true[g] = fmaxf(m_true[g], tile_max(sc[g]));
    } else {
      if (t == 0 && set_ref) {
#pragma unroll
        for (int g = 0; g < NG; ++g) {
          const float tmax = tile_max(sc[g]);
          m_ref[g] = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
        }
      }
      bf16x8 pp[NG][2];
      softmax(sc, pp);
      __builtin_amdgcn_sched_barrier(0);
      pv_acc(VS, pp);
    }
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  // One pass over the item's key tiles in the given mode.
  auto key_pass = [&](auto mode_t, bool set_ref, bool first_pass) __attribute__((always_inline)) {
    constexpr int MODE = decltype(mode_t)::value;
    if constexpr (MODE == 0) {
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        l_run[g] = 0.f;
#pragma unroll
        for (int n = 0; n < NT; ++n)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[g][n][r] = 0.f;
      }
    }
    // Prologue: K tile 0, V tile 0, K tile 1 (then Q on the first pass, all in
    // flight together).
    copy_tile(0, pk, ak, kstage(0));
    copy_tile(0, pv, av, vstage(0));
    copy_tile(1, pk, ak, kstage(1));
    if (first_pass) {
      load_q();
      // Wait here for Q (and so for the copies issued before it): the key
      // loop then holds no wait for loads the compiler knows of, which would
      // also wait for the copies issued inside the loop.
#pragma unroll
      for (int g = 0; g < NG; ++g)
#pragma unroll
        for (int i = 0; i < NS; ++i) asm volatile("" : "+v"(qf[g][i]));
    }
    step(0, I0{}, I0{}, mode_t, set_ref);
    // Steps 1 .. nkt - 1, six per round (the period of the two rings).
    for (int t = 1; t < nkt;) {
      step(t, I1{}, I1{}, mode_t, false);
      if (++t >= nkt) break;
      step(t, I2{}, I0{}, mode_t, false);
      if (++t >= nkt) break;
      step(t, I0{}, I1{}, mode_t, false);
      if (++t >= nkt) break;
      step(t, I1{}, I0{}, mode_t, false);
      if (++t >= nkt) break;
      step(t, I2{}, I1{}, mode_t, false);
      if (++t >= nkt) break;
      step(t, I0{}, I0{}, mode_t, false);
      ++t;
    }
    __builtin_amdgcn_s_waitcnt(at::waitcnt_vm(0));   // no copy may outlive the pass (or the block's LDS)
    __syncthreads();                                 // every wave's copies have landed and its reads are done
  };

  // First pass against the first tile's maxima.  If any wave saw a sum
  // overflow, the block takes the true maxima in a second pass and runs the
  // item again against them (every P <= 1 then).
  key_pass(I0{}, true, true);
  {
    uint32_t *vote = reinterpret_cast<uint32_t *>(smem);
    const bool any = __ballot(ovf != 0) != 0;
    if (lane == 0) vote[wave] = any ? 1u : 0u;
    __syncthreads();
    const uint32_t again = vote[0] | vote[1] | vote[2] | vote[3];
    __syncthreads();                                 // the votes are read before the copies refill the rings
    if (again) {
      key_pass(I1{}, false, false);
#pragma unroll
      for (int g = 0; g < NG; ++g) m_ref[g] = fmaxf(m_true[g], __shfl_xor(m_true[g], 32, 64));
      key_pass(I0{}, false, false);
    }
  }

  // Accumulator layout: lane holds query (lane & 31) of the group; register r
  // of tile n holds head-dim index 32 n + (r/4)*8 + 4 half + r%4.
  constexpr int CPRO = HD / 8;              // 16-byte chunks per output row
  __syncthreads();                          // every wave is done with the rings
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const float l_all = l_run[g] + __shfl_xor(l_run[g], 32, 64);
    const int loc = 32 * (wave + 4 * g) + (lane & 31);
    if (loc >= it.nq) continue;
    if (it.slot < 0) {
      // Through LDS (the rings, free now): lane q writes its query row's 8-byte
      // pieces, chunk c of a row at c ^ (q % CPRO); then rows go out as whole
      // 16-byte chunks, consecutive lanes on consecutive chunks of a row.
      const float inv = 1.0f / l_all;
      uint8_t *stg = smem + (wave * NG + g) * (32 * 2 * HD);
      const int q = lane & 31;
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          bf16x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = (bf16)(o[g][n][rg * 4 + e] * inv);
          const int c = (4 * n + rg) ^ (q & (CPRO - 1));
          *reinterpret_cast<bf16x4 *>(stg + q * 2 * HD + c * 16 + half * 8) = v;
        }
    }
  }
  __builtin_amdgcn_s_waitcnt(at::waitcnt_lgkm0);   // this wave's staging writes are done
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int base = 32 * (wave + 4 * g);
    if (it.slot >= 0 || base >= it.nq) continue;
    const uint8_t *stg = smem + (wave * NG + g) * (32 * 2 * HD);
    constexpr int RPI = 64 / CPRO;          // rows per instruction
#pragma unroll
    for (int i = 0; i < 32 / RPI; ++i) {
      const int r = i * RPI + lane / CPRO, c = lane % CPRO;
      if (base + r < it.nq) {
        const int qrow = it.q0 + base + r;
        const uint4 v = *reinterpret_cast<const uint4 *>(stg + r * 2 * HD + ((c ^ (r & (CPRO - 1))) * 16));
        const size_t orow = (size_t)(it.tok_off + qrow / G), ocol = (size_t)(it.kvh * G + qrow % G) * HD + c * 8;
        // row-major, or kb32 (the 16-byte chunk stays inside one 32-wide block)
        const size_t off = a.o_rows > 0 ? kb32_offset(a.o_rows, orow, ocol) : orow * a.ldo + ocol;
        *reinterpret_cast<uint4 *>(reinterpret_cast<bf16 *>(a.o) + off) = v;
      }
    }
  }
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const float l_all = l_run[g] + __shfl_xor(l_run[g], 32, 64);
    const int loc = 32 * (wave + 4 * g) + (lane & 31);
    if (loc >= it.nq) continue;
    if (it.slot >= 0) {
      bf16 *po = reinterpret_cast<bf16 *>(a.part_o) + ((size_t)it.slot * kAttnQB + loc) * HD;
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          bf16x4 v;
#pragma unroll
          for (int e2 = 0; e2 < 4; ++e2) v[e2] = (bf16)o[g][n][rg * 4 + e2];
          *reinterpret_cast<bf16x4 *>(po + n * 32 + rg * 8 + half * 4) = v;
        }
      if (half == 0) {
        float *pm = a.part_ml + ((size_t)it.slot * kAttnQB + loc) * 2;
        pm[0] = m_ref[g] * sl2;     // log2 units, as the merge expects
        pm[1] = l_all;
      }
    }
  }
  __syncthreads();                          // the staging reads are done before the next item's copies
  }
}

// ------------------------------------------------------------------ fp32 attention (debug mode)
// One wave per query row, keys in order, online softmax; lanes own head-dim
// elements.  Slow and simple.
template <int HD>
__global__ void __launch_bounds__(256) attention_f32_kernel(AttnArgs a) {
  constexpr int EPL = (HD + 63) / 64;   // head-dim elements per lane
  const AttnItem it = a.items[blockIdx.x];
  const ReqDesc rq = a.reqs[it.req];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int G = a.nq / a.nkv;
  const int qloc = blockIdx.y * 4 + wave;
  if (qloc >= it.nq) return;
  const int qrow = it.q0 + qloc;
  const int qt = qrow / G, qg = it.kvh * G + qrow % G;
  const float *qkv = reinterpret_cast<const float *>(a.qkv);
  const float *qp = qkv + (size_t)(rq.tok_off + qt) * a.ldqkv + (size_t)qg * HD;
  const size_t prow = (size_t)a.nkv * HD;
  const float *pk = reinterpret_cast<const float *>(rq.pk) + (size_t)a.layer * rq.P * prow + (size_t)it.kvh * HD;
  const float *pv = reinterpret_cast<const float *>(rq.pv) + (size_t)a.layer * rq.P * prow + (size_t)it.kvh * HD;
  const float *ak = qkv + (size_t)rq.tok_off * a.ldqkv + (size_t)(a.nq + it.kvh) * HD;
  const float *av = qkv + (size_t)rq.tok_off * a.ldqkv + (size_t)(a.nq + a.nkv + it.kvh) * HD;
  float q[EPL], acc[EPL];
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const int e = lane + 64 * j;
    q[j] = e < HD ? qp[e] : 0.f;
    acc[j] = 0.f;
  }
  const float scale = 1.0f / sqrtf((float)HD);
  float m = -INFINITY, l = 0.f;
  const int kend = a.causal ? min(it.kend, max(it.causal_b, qt + 1)) : it.kend;
  for (int key = it.kbeg; key < kend; ++key) {
    const float *kr = key < rq.P ? pk + (size_t)key * prow : ak + (size_t)(key - rq.P) * a.ldqkv;
    const float *vr = key < rq.P ? pv + (size_t)key * prow : av + (size_t)(key - rq.P) * a.ldqkv;
    float dot = 0.f;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const int e = lane + 64 * j;
      if (e < HD) dot = fmaf(q[j], kr[e], dot);
    }
    dot = wave_sum(dot) * scale;
    const float m_new = fmaxf(m, dot);
    const float alpha = expf(m - m_new);
    const float p = expf(dot - m_new);
    l = l * alpha + p;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const int e = lane + 64 * j;
      acc[j] = acc[j] * alpha + (e < HD ? p * vr[e] : 0.f);
    }
    m = m_new;
  }
  float *op = reinterpret_cast<float *>(a.o) + (size_t)(rq.tok_off + qt) * a.ldo + (size_t)qg * HD;
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const int e = lane + 64 * j;
    if (e < HD) op[e] = acc[j] / l;
  }
}

// ------------------------------------------------------------------ merge of split-key partials
// One wave per query row of a split group: combine the group's partials in
// slot order: m = max_c m_c, w_c = 2^(m_c - m), o = sum_c w_c O_c / sum_c w_c l_c
// (O_c in bf16, m_c and l_c in fp32).
template <typename OutT>
__global__ void __launch_bounds__(256) attn_merge_kernel(const AttnGroup *__restrict__ groups,
                                                         const ReqDesc *__restrict__ reqs,
                                                         const bf16 *__restrict__ part_o,
                                                         const float *__restrict__ part_ml, OutT *o,
                                                         int ldo, int nq, int nkv, int hd, int o_rows) {
  const AttnGroup gr = groups[blockIdx.y];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int qloc = blockIdx.x * 4 + wave;
  const int G = nq / nkv;
  if (qloc >= gr.nq) return;
  const int tok_off = reqs[gr.req].tok_off;   // issued now, used for the store
  const int qrow = gr.q0 + qloc;
  const int qt = qrow / G, qg = gr.kvh * G + qrow % G;
  // Partials are read CH slots at a time (their max and sum with their O),
  // every load of a batch in flight together, so a group of at most CH
  // slots costs one round trip; batches combine in slot order against a
  // running max (the sums so far rescaled when a later batch raises it).
  // Lane holds head-dim elements 4 lane .. 4 lane + 3 (head_dim <= 256).
  constexpr int CH = 8;
  const int e0 = lane * 4;
  const bool on = e0 < hd;
  const float2 *ml = reinterpret_cast<const float2 *>(part_ml);
  float mx = -INFINITY, L = 0.f;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int c0 = 0; c0 < gr.n; c0 += CH) {
    float2 p[CH];
    bf16x4 ov[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const size_t base = (size_t)(gr.first_slot + c0 + c) * kAttnQB + qloc;
      const bool live = c0 + c < gr.n;
      p[c] = live ? ml[base] : make_float2(-INFINITY, 0.f);
      ov[c] = live && on ? *reinterpret_cast<const bf16x4 *>(part_o + base * hd + e0) : bf16x4{};
    }
    float nm = mx;
#pragma unroll
    for (int c = 0; c < CH; ++c) nm = fmaxf(nm, p[c].x);
    const float sc = exp2f(mx - nm);          // 0 on the first batch (mx = -inf)
    L *= sc;
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] *= sc;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      if (c0 + c >= gr.n) break;
      const float wgt = exp2f(p[c].x - nm);
      L += wgt * p[c].y;
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] += wgt * (float)ov[c][j];
    }
    mx = nm;
  }
  if (!on) return;
  const float inv = 1.0f / L;
  const size_t orow = (size_t)(tok_off + qt), col = (size_t)qg * hd + e0;
  OutT *dst = o + (o_rows > 0 ? kb32_offset(o_rows, orow, col) : orow * ldo + col);
#pragma unroll
  for (int j = 0; j < 4; ++j) dst[j] = from_f32<OutT>(acc[j] * inv);
}


hipError_t launch_attention(const AttnArgs &a, bool bf16_mode, hipStream_t s) {
  if (a.n_items <= 0) return hipSuccess;
  if (a.o_rows > 0 && !bf16_mode) return hipErrorInvalidValue;
  if (bf16_mode) {
    if (a.n_blocks <= 0) return hipSuccess;
    dim3 grid(a.n_blocks);
    switch (a.hd) {
      case 32:
        if (a.causal) hipLaunchKernelGGL((attention_bf16_kernel<32, attn_groups_per_wave(32), true>), grid, dim3(256), 0, s, a);
        else hipLaunchKernelGGL((attention_bf16_kernel<32, attn_groups_per_wave(32), false>), grid, dim3(256), 0, s, a);
        break;
      case 64:
        if (a.causal) hipLaunchKernelGGL((attention_bf16_kernel<64, attn_groups_per_wave(64), true>), grid, dim3(256), 0, s, a);
        else hipLaunchKernelGGL((attention_bf16_kernel<64, attn_groups_per_wave(64), false>), grid, dim3(256), 0, s, a);
        break;
      case 128:
        if (a.causal) hipLaunchKernelGGL((attention_bf16_kernel<128, attn_groups_per_wave(128), true>), grid, dim3(256), 0, s, a);
        else hipLaunchKernelGGL((attention_bf16_kernel<128, attn_groups_per_wave(128), false>), grid, dim3(256), 0, s, a);
        break;
      case 256:
        if (a.causal) hipLaunchKernelGGL((attention_bf16_kernel<256, attn_groups_per_wave(256), true>), grid, dim3(256), 0, s, a);
        else hipLaunchKernelGGL((attention_bf16_kernel<256, attn_groups_per_wave(256), false>), grid, dim3(256), 0, s, a);
        break;
      default: return hipErrorInvalidValue;
    }
  } else {
    dim3 grid(a.n_items, kAttnQB / 4);
    switch (a.hd) {
      case 32: hipLaunchKernelGGL(attention_f32_kernel<32>, grid, dim3(256), 0, s, a); break;
      case 64: hipLaunchKernelGGL(attention_f32_kernel<64>, grid, dim3(256), 0, s, a); break;
      case 128: hipLaunchKernelGGL(attention_f32_kernel<128>, grid, dim3(256), 0, s, a); break;
      case 256: hipLaunchKernelGGL(attention_f32_kernel<256>, grid, dim3(256), 0, s, a); break;
      default: return hipErrorInvalidValue;
    }
  }
  return hipGetLastError();
}

hipError_t launch_attn_merge(const AttnGroup *groups, int n_groups, const ReqDesc *reqs,
                             const void *part_o, const float *part_ml, void *o, int ldo, int nq,
                             int nkv, int hd, bool bf16_mode, hipStream_t s, int o_rows) {
  if (n_groups <= 0) return hipSuccess;
  if (hd > 256) return hipErrorInvalidValue;   // a lane holds at most 4 head-dim elements
  if (o_rows > 0 && !bf16_mode) return hipErrorInvalidValue;
  dim3 grid(kAttnQB / 4, n_groups);
  if (bf16_mode)
    hipLaunchKernelGGL(attn_merge_kernel<bf16>, grid, dim3(256), 0, s, groups, reqs, (const bf16 *)part_o, part_ml,
                       (bf16 *)o, ldo, nq, nkv, hd, o_rows);
  else
    hipLaunchKernelGGL(attn_merge_kernel<float>, grid, dim3(256), 0, s, groups, reqs, (const bf16 *)part_o, part_ml,
                       (float *)o, ldo, nq, nkv, hd, 0);
  return hipGetLastError();
}

}  // namespace rosa
