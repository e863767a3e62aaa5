// Ragged prefix + action attention of one layer.
//
// Request r's H_r action tokens (G = n_q / n_kv query heads per KV head, so
// G*H_r query rows per KV head) attend to its own key sequence: the P_r cached
// prefix keys of this layer followed by its H_r action keys; no other request
// and no padding is visible.  Scale 1/sqrt(head_dim); no causal mask.
//
// bf16 kernel (gfx950 MFMA).  A work item is (request, KV head, up to 128 NG
// query rows, key range).  Its four waves stream the key range through LDS in
// 32-key tiles: a K ring and a V ring of four stages each, filled by
// global_load_lds_dwordx4 with two copy groups in flight.  Each wave owns NG
// groups of 32 query rows (groups w and w + 4 of the item), so every K and V
// fragment it reads from LDS feeds the MFMAs of all its groups; NG is 2 where
// Q^T and O^T of two groups fit the register file (head_dim <= 128) and 1
// otherwise.  Step t computes S^T = K Q^T of tile t with
// v_mfma_f32_32x32x16_bf16 (K from LDS, Q^T held in registers for the whole
// item; each lane owns one query column, so softmax statistics are in-lane)
// and O^T += V^T P^T of tile t - 1 (P^T from registers, V^T from the
// row-major V tile through the LDS transpose read ds_read_b64_tr_b16), with
// the softmax of tile t interleaved between the PV MFMAs.  Every MFMA's LDS
// operand is read two fragments ahead.  The softmax uses a fixed reference
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
constexpr int kChains = 2;          // independent S accumulator chains (even / odd k-steps)
constexpr bool kSpreadCopies = false; // copies spread over the step, else in the first slots
}  // namespace at

#define ROSA_LDS_A(p) ((__attribute__((address_space(3))) void *)(p))


// One 1 KB global -> LDS copy (lane i: 16 bytes from its own source to
// lds + 16 i), written as inline assembly so the compiler does not track it:
// its model of this copy makes it wait for every outstanding LDS read before
// the next MFMA, which would cap the LDS reads in flight at one.  The kernel
// waits for the copies itself (vmcnt) and sets M0, which nothing else in these
// kernels uses; the s_nop is the wait state the M0 write needs before the copy.
__device__ __forceinline__ void dma_1k(const void *src, uint32_t lds) {
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds) : "memory", "m0");
#pragma clang diagnostic pop
}
__device__ __forceinline__ uint32_t lds_u32(const uint8_t *p) {
  return (uint32_t)(size_t)ROSA_LDS_A(p);
}
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
template <int HD>
struct AttnTile {
  static constexpr int ROWB = HD * 2;             // bytes per K or V row
  static constexpr int CPR = ROWB / 16;           // 16-byte chunks per row
  static constexpr int TILEB = 32 * ROWB;         // bytes of one 32-key K (or V) tile
  static constexpr int UNITS = 2 * TILEB / 1024;  // 1 KB copies per stage (K then V)
  static constexpr int CPW = 2 * ((UNITS / 2 + 3) / 4);   // copies per copying wave per stage
  static constexpr int RPU = 1024 / ROWB;         // rows per 1 KB copy
  // A wave copies CPW units of a stage or none, so waiting until at most
  // 2 CPW copies are outstanding leaves exactly the two next stages in flight.
  static constexpr int WAIT = at::waitcnt_vm(2 * CPW);
  static constexpr int WAIT0 = at::waitcnt_vm(0);
  static_assert((UNITS / 2) % 4 == 0 || UNITS / 2 < 4, "copy split");
};

template <int HD, int NG>
__global__ void __launch_bounds__(256, 1) attention_bf16_kernel(AttnArgs a) {
  using at::TK;
  using T = AttnTile<HD>;
  constexpr int NS = HD / 16;       // MFMA k-steps over head_dim for S
  constexpr int NT = HD / 32;       // 32-row output tiles over head_dim
  constexpr int NF = NS + 2 * NT;   // LDS operand fragments (and MFMA slots) per step
  constexpr int CPR = T::CPR, ROWB = T::ROWB, TILEB = T::TILEB;
  // K ring and V ring of four 32-key tiles each: K stage s at s TILEB, V
  // stage s at (4 + s) TILEB.  Step t computes S for tile t and O += P V for
  // tile t - 1, so the V ring runs one tile behind the K ring.  Every stage
  // offset from a ring's lane base fits a ds_read immediate.
  __shared__ __attribute__((aligned(1024))) uint8_t smem[8 * TILEB];
  static_assert(4 * TILEB <= 65536, "stage offsets must fit the LDS immediate");

  const AttnItem it = a.ordered[blockIdx.x];
  if (it.nq <= 0) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & 3;   // wave-uniform, in an SGPR
  const int half = lane >> 5;
  const int G = a.nq / a.nkv;
  const bf16 *qkv = reinterpret_cast<const bf16 *>(a.qkv);

  // Q^T operand of group g, held for the whole item: lane holds
  // Q[row][16 s + 8 half .. + 7] for its row; rows past the item's queries
  // read the item's first row instead (their results are never stored).
  // Loaded right after the first copy group is issued, so the two latencies
  // overlap: the compiler does not see the copies, and its wait for Q (all
  // loads it knows of) then also covers the copy group issued before it.
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
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
      for (int s = 0; s < NS; ++s) asm volatile("" : "+v"(qf[g][s]));
  };

  const size_t prow = (size_t)a.nkv * HD;   // prefix row stride (elements)
  const bf16 *pk = reinterpret_cast<const bf16 *>(it.pk) + (size_t)a.layer * it.P * prow + (size_t)it.kvh * HD;
  const bf16 *pv = reinterpret_cast<const bf16 *>(it.pv) + (size_t)a.layer * it.P * prow + (size_t)it.kvh * HD;
  const bf16 *ak = qkv + (size_t)it.tok_off * a.ldqkv + (size_t)(a.nq + it.kvh) * HD;
  const bf16 *av = qkv + (size_t)it.tok_off * a.ldqkv + (size_t)(a.nq + a.nkv + it.kvh) * HD;
  const long ldq = a.ldqkv;
  // Tile t covers keys [k0 + 32 t, k0 + 32 t + 32) with k0 = kend - 32 nkt:
  // only tile 0 can reach below kbeg (those keys are masked), so the key
  // loop itself never masks.
  const int nkt = (it.kend - it.kbeg + TK - 1) / TK;
  const int k0 = it.kend - TK * nkt;
  const uint32_t lds0 = lds_u32(smem);

  // Copies: 1 KB units, unit u of a tile by wave u % 4; lane i fills physical
  // chunk i % CPR of row u * RPU + i / CPR, which holds logical chunk
  // (i % CPR) ^ swz(row).  Keys below the range load the first valid key
  // (finite values; their scores are masked).  A tile that lies wholly in the
  // prefix (all but at most three per item) takes its sources from a uniform
  // base plus per-lane offsets fixed for the whole item; the others compute
  // each lane's key.  Tile indices past the last tile copy the last tile
  // again (harmless: that stage is not in use).
  constexpr int UPW = (T::UNITS / 2 + 3) / 4;    // units of one tile per copying wave
  constexpr int NCP = 2 * UPW;                   // copies per group (K units, then V units)
  int poff[UPW];
#pragma unroll
  for (int j = 0; j < UPW; ++j) {
    const int row = (4 * j + wave) * T::RPU + lane / CPR;
    poff[j] = row * (int)prow + (((lane % CPR) ^ at::swz(row, CPR)) << 3);
  }
  struct TileSrc {
    const bf16 *lane[UPW];
  };
  auto sources = [&](int t, const bf16 *pbase, const bf16 *abase, TileSrc &ts) __attribute__((always_inline)) {
    const int kt0 = k0 + max(0, min(t, nkt - 1)) * TK;
    if (kt0 >= it.kbeg && kt0 + TK <= it.P) {
      const bf16 *b = pbase + (size_t)kt0 * prow;
#pragma unroll
      for (int j = 0; j < UPW; ++j) ts.lane[j] = b + poff[j];
    } else {
      // Recomputed from an opaque copy of the lane index at every use, so the
      // compiler does not hoist these per-lane addresses out of the key loop
      // (they would hold registers for the whole loop).
      int ln = lane;
      asm volatile("" : "+v"(ln));
#pragma unroll
      for (int j = 0; j < UPW; ++j) {
        const int row = (4 * j + wave) * T::RPU + ln / CPR;
        const int c = (ln % CPR) ^ at::swz(row, CPR);
        const int key = max(kt0 + row, it.kbeg);
        const bool pre = key < it.P;
        const long roff = (pre ? (long)key * (long)prow : (long)(key - it.P) * ldq) + c * 8;
        ts.lane[j] = (pre ? pbase : abase) + roff;
      }
    }
  };
  // Copy c of a group: K tile -> K stage kst (c < UPW), V tile -> V stage vst.
  auto copy = [&](const TileSrc &k, const TileSrc &v, int kst, int vst, int c) __attribute__((always_inline)) {
    const int j = c % UPW;
    if (4 * j + wave >= T::UNITS / 2) return;
    const uint32_t dst = lds0 + (c < UPW ? kst : 4 + vst) * TILEB + (4 * j + wave) * 1024;
    dma_1k(c < UPW ? k.lane[j] : v.lane[j], dst);
  };

  // K operand: row lane%32, logical chunk 2 ks + half.  The swizzle touches
  // the low four chunk bits only, so k-steps 8 apart differ by 256 bytes.
  const int krow = lane & 31;
  constexpr int NKO = NS < 8 ? NS : 8;
  uint32_t kb[NKO];
#pragma unroll
  for (int i = 0; i < NKO; ++i) {
    kb[i] = lds0 + krow * ROWB + (((2 * i + half) ^ at::swz(krow, CPR)) << 4);
    asm volatile("" : "+v"(kb[i]));   // a lane base: stage offsets become immediates
  }
  // V transpose reads: source lane s of 16-lane group G16 reads 8 bytes at
  // row 16 ks + 4 half + s/4 (and 8 rows further), head-dim column
  // 32 n + 16 G16 + 4 (s%4).  The row's swizzle does not depend on ks, and
  // output tiles 4 apart differ by 256 bytes.
  const int src16 = lane & 15, g16 = (lane >> 4) & 1;
  const int vcol = 16 * g16 + 4 * (src16 & 3);
  constexpr int NVO = NT < 4 ? NT : 4;
  uint32_t vb[2][NVO];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int r = half * 4 + (src16 >> 2) + 8 * h;
    const int sw = at::swz(r, CPR);
#pragma unroll
    for (int n = 0; n < NVO; ++n) {
      const int x = n * 32 + vcol;
      vb[h][n] = lds0 + 4 * TILEB + r * ROWB + (((x >> 3) ^ sw) << 4) + ((x & 7) << 1);
      asm volatile("" : "+v"(vb[h][n]));
    }
  }
  // Fragment j of a step (K stage ks, V stage vs): j < NS is K k-step j (S^T
  // operand); the others are V^T k-step (j - NS) / NT, output tile (j - NS) % NT.
  auto load_frag = [&](int kst, int vst, int j) __attribute__((always_inline)) -> bf16x8 {
    if (j < NS) return *reinterpret_cast<const __attribute__((address_space(3))) bf16x8 *>(lds_ptr(kb[j % 8]) + kst * TILEB + (j / 8) * 256);
    const int ks = (j - NS) / NT, n = (j - NS) % NT;
    const int c = vst * TILEB + (n / 4) * 256 + ks * 16 * ROWB;
    return lds_tr_pair(lds_ptr(vb[0][n % 4]) + c, lds_ptr(vb[1][n % 4]) + c);
  };

  f32x16 o[NG][NT];
  // Softmax without rescaling the output inside the key loop: each query's
  // reference max m_ref is its max over the item's first 32-key tile, and
  // P = 2^((s - m_ref) log2(e) / sqrt(hd)) may exceed 1.  The loop tracks the
  // true max; if any query's later scores exceed its reference by more than
  // 2^64 (room to spare below fp32 overflow for the sums), the block runs the
  // item a second time with the true max as reference, where P <= 1.  Either
  // way the output accumulators are only touched by MFMAs in the loop.  The
  // two 32-lane halves hold different keys of the same query: after the first
  // tile they keep their own running max and sum, combined at the end.
  float m_ref[NG], m_true[NG], l_run[NG], mb[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) m_true[g] = -INFINITY;
  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);   // log2(e) / sqrt(hd)
  const float over = 64.0f / sl2;           // raw score excess that asks for the second pass
  int ovf = 0;

  // One step = NF slots in a fixed order (sched_barrier fences keep the
  // compiler from regrouping them): slot j issues the LDS read of fragment
  // j + 2 and the MFMAs of fragment j, so every MFMA finds its operand two
  // reads ahead.  S^T (32 keys x 32 queries; lane = query lane%32, register
  // r = key (r/4)*8 + 4 half + r%4) accumulates in kChains independent MFMA
  // chains per group (k-steps alternate between them).  The copies
  // of the next group are spread evenly over the slots; the softmax of this
  // tile (P^T for the next step) fills the PV slots from slot NS + 1.
  bf16x8 pp[NG][2];   // P^T of the previous tile: PV k-step ks uses registers 8 ks .. 8 ks + 7
  auto run_step = [&](auto has_s_t, auto has_pv_t, int t, int kst, int vst, int kref, int vref)
                      __attribute__((always_inline)) {
    constexpr bool HAS_S = decltype(has_s_t)::value, HAS_PV = decltype(has_pv_t)::value;
    constexpr bool COPY = HAS_S && HAS_PV;
    constexpr int J0 = HAS_S ? 0 : NS, J1 = HAS_PV ? NF : NS;
    constexpr int CSTRIDE = at::kSpreadCopies ? NF / NCP : 1;   // slots between copies
    TileSrc ksrc, vsrc;
    if constexpr (COPY) {
      sources(t + 3, pk, ak, ksrc);
      sources(t + 2, pv, av, vsrc);
    }
    f32x16 s[NG][at::kChains];
    float tmax[NG], psum[NG];
    bf16x8 pn[NG][2];
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
      for (int c = 0; c < at::kChains; ++c)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[g][c][r] = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) { tmax[g] = -INFINITY; psum[g] = 0.f; }
    // Softmax of scores r, r + 1 of group g (a step after the first tile).
    auto soft_pair = [&](int g, int r) __attribute__((always_inline)) {
      float x0 = s[g][0][r], x1 = s[g][0][r + 1];
      if (at::kChains == 2) { x0 += s[g][1][r]; x1 += s[g][1][r + 1]; }
      tmax[g] = fmaxf(tmax[g], fmaxf(x0, x1));
      const float e0 = __builtin_amdgcn_exp2f(fmaf(x0, sl2, mb[g]));
      const float e1 = __builtin_amdgcn_exp2f(fmaf(x1, sl2, mb[g]));
      psum[g] += e0;
      psum[g] += e1;
      pn[g][r >> 3][r & 7] = (bf16)e0;
      pn[g][r >> 3][(r & 7) + 1] = (bf16)e1;
      // Keep the work in this slot: the values are only used a step later,
      // and the compiler would otherwise move it next to that use.
      asm volatile("" : "+v"(pn[g][r >> 3]), "+v"(psum[g]), "+v"(tmax[g]));
    };
    constexpr int NPAIR = 8 * NG;                        // score pairs per tile
    constexpr int SOFT0 = NS + 1;                        // first slot that takes softmax work
    constexpr int NSOFT = NF - SOFT0;                    // slots that take it
    bf16x8 fr[3];
#pragma unroll
    for (int j = J0; j < J0 + 2 && j < J1; ++j) fr[j % 3] = load_frag(kst, vst, j);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = J0; j < J1; ++j) {
      if (j + 2 < J1) fr[(j + 2) % 3] = load_frag(kst, vst, j + 2);
      if (COPY && j % CSTRIDE == 0 && j / CSTRIDE < NCP) copy(ksrc, vsrc, kref, vref, j / CSTRIDE);
      if (j < NS) {
#pragma unroll
        for (int g = 0; g < NG; ++g) {
          f32x16 &acc = s[g][j % at::kChains];
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[j % 3], qf[g][j], acc, 0, 0, 0);
        }
      } else {
        const int ks = (j - NS) / NT, n = (j - NS) % NT;
#pragma unroll
        for (int g = 0; g < NG; ++g) o[g][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[j % 3], pp[g][ks], o[g][n], 0, 0, 0);
        if (HAS_S && j >= SOFT0) {
          // pairs [p0, p1) of this slot, spread evenly over the softmax slots
          const int p0 = (j - SOFT0) * NPAIR / NSOFT, p1 = (j - SOFT0 + 1) * NPAIR / NSOFT;
#pragma unroll
          for (int p = p0; p < p1; ++p) soft_pair(p / 8, 2 * (p % 8));
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (HAS_S && HAS_PV) {
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        m_true[g] = fmaxf(m_true[g], tmax[g]);
        ovf |= tmax[g] > m_ref[g] + over;
        l_run[g] += psum[g];
        pp[g][0] = pn[g][0];
        pp[g][1] = pn[g][1];
      }
    }
  };
  // The first tile: S, then its softmax whole (it may set the reference max
  // and carries the mask of keys below the range).
  auto first_tile = [&](bool set_ref) __attribute__((always_inline)) {
    f32x16 s[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[g][r] = 0.f;
#pragma unroll
    for (int ks = 0; ks < NS; ++ks) {
      const bf16x8 kf = load_frag(0, 0, ks);
#pragma unroll
      for (int g = 0; g < NG; ++g) s[g] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[g][ks], s[g], 0, 0, 0);
    }
#pragma unroll
    for (int g = 0; g < NG; ++g) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = k0 + (r >> 2) * 8 + half * 4 + (r & 3);
        if (key < it.kbeg) s[g][r] = -INFINITY;
      }
      float tmax = s[g][0];
#pragma unroll
      for (int r = 1; r < 16; ++r) tmax = fmaxf(tmax, s[g][r]);
      if (set_ref) m_ref[g] = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
      mb[g] = -m_ref[g] * sl2;
      m_true[g] = fmaxf(m_true[g], tmax);
      ovf |= tmax > m_ref[g] + over;
      float ps = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float pe = __builtin_amdgcn_exp2f(fmaf(s[g][r], sl2, mb[g]));
        ps += pe;
        pp[g][r >> 3][r & 7] = (bf16)pe;
      }
      l_run[g] += ps;
    }
  };

  for (int pass = 0; pass < 2; ++pass) {
    const bool pass0 = pass == 0;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      l_run[g] = 0.f;
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[g][n][r] = 0.f;
    }
    // Step t (1 <= t < nkt): wait for copy group t, refill with group t + 3
    // (K tile t + 3 into the stage K tile t - 1 left, V tile t + 2 into the
    // stage V tile t - 2 left), S of tile t, O += P V of tile t - 1, P of
    // tile t.  Copy group j = K tile j and V tile j - 1.
    auto step = [&](int t, int kst, int vst, int kref, int vref) __attribute__((always_inline)) {
      __builtin_amdgcn_s_waitcnt(T::WAIT);    // this wave's copies of group t have landed
      __builtin_amdgcn_s_barrier();           // ... and every wave's; the refilled stages are free
      __builtin_amdgcn_sched_barrier(0);
      run_step(std::true_type{}, std::true_type{}, t, kst, vst, kref, vref);
    };
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      TileSrc ksrc, vsrc;
      sources(j, pk, ak, ksrc);
      sources(j - 1, pv, av, vsrc);
#pragma unroll
      for (int c = 0; c < NCP; ++c) copy(ksrc, vsrc, j, (j + 3) & 3, c);
      if (j == 0 && pass0) load_q();        // lands with copy group 0
    }
    {   // step 0: S and P of the first tile, refill with group 3
      __builtin_amdgcn_s_waitcnt(T::WAIT);
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      TileSrc ksrc, vsrc;
      sources(3, pk, ak, ksrc);
      sources(2, pv, av, vsrc);
#pragma unroll
      for (int c = 0; c < NCP; ++c) copy(ksrc, vsrc, 3, 2, c);
      first_tile(pass0);
    }
    // Whole groups of four steps, then the last one to three steps.
    int t = 1;
    for (; t + 4 <= nkt; t += 4) {
      step(t, 1, 0, 0, 3);
      step(t + 1, 2, 1, 1, 0);
      step(t + 2, 3, 2, 2, 1);
      step(t + 3, 0, 3, 3, 2);
    }
    if (t < nkt) {
      step(t, 1, 0, 0, 3);
      if (t + 1 < nkt) {
        step(t + 1, 2, 1, 1, 0);
        if (t + 2 < nkt) step(t + 2, 3, 2, 2, 1);
      }
    }
    // O += P V of the last tile, once every copy has landed.
    __builtin_amdgcn_s_waitcnt(T::WAIT0);   // no copy may outlive the pass (or the block's LDS)
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    switch ((nkt - 1) & 3) {
      case 0: run_step(std::false_type{}, std::true_type{}, 0, 0, 0, 0, 0); break;
      case 1: run_step(std::false_type{}, std::true_type{}, 0, 0, 1, 0, 0); break;
      case 2: run_step(std::false_type{}, std::true_type{}, 0, 0, 2, 0, 0); break;
      default: run_step(std::false_type{}, std::true_type{}, 0, 0, 3, 0, 0); break;
    }
    // Block-uniform decision: every wave has finished reading the stages.
    if (!pass0 || !__syncthreads_or(ovf)) break;
#pragma unroll
    for (int g = 0; g < NG; ++g) m_ref[g] = fmaxf(m_true[g], __shfl_xor(m_true[g], 32, 64));
  }

  // Accumulator layout: lane holds query (lane & 31) of the group; register r
  // of tile n holds head-dim index 32 n + (r/4)*8 + 4 half + r%4.
  constexpr int CPRO = HD / 8;              // 16-byte chunks per output row
  static_assert(4 * NG * 32 * 2 * HD <= 8 * TILEB, "output staging fits the rings");
  __syncthreads();                          // every wave is done with the rings
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const float l_all = l_run[g] + __shfl_xor(l_run[g], 32, 64);
    const int loc = 32 * (wave + 4 * g) + (lane & 31);
    if (loc >= it.nq) continue;
    if (it.slot < 0) {
      // Through LDS (the K ring, free now): lane q writes its query row's 8-byte
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
        bf16 *op = reinterpret_cast<bf16 *>(a.o) + (size_t)(it.tok_off + qrow / G) * a.ldo +
                   (size_t)(it.kvh * G + qrow % G) * HD;
        *reinterpret_cast<uint4 *>(op + c * 8) = v;
      }
    }
  }
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const float l_all = l_run[g] + __shfl_xor(l_run[g], 32, 64);
    const int loc = 32 * (wave + 4 * g) + (lane & 31);
    if (loc >= it.nq) continue;
    if (it.slot >= 0) {
      float *po = a.part_o + ((size_t)it.slot * kAttnQB + loc) * HD;
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const float4 v = make_float4(o[g][n][rg * 4 + 0], o[g][n][rg * 4 + 1], o[g][n][rg * 4 + 2], o[g][n][rg * 4 + 3]);
          *reinterpret_cast<float4 *>(po + n * 32 + rg * 8 + half * 4) = v;
        }
      if (half == 0) {
        float *pm = a.part_ml + ((size_t)it.slot * kAttnQB + loc) * 2;
        pm[0] = m_ref[g] * sl2;     // log2 units, as the merge expects
        pm[1] = l_all;
      }
    }
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
  for (int key = it.kbeg; key < it.kend; ++key) {
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
// slot order: m = max_c m_c, w_c = 2^(m_c - m), o = sum_c w_c O_c / sum_c w_c l_c.
template <typename OutT>
__global__ void __launch_bounds__(256) attn_merge_kernel(const AttnGroup *__restrict__ groups,
                                                         const ReqDesc *__restrict__ reqs,
                                                         const float *__restrict__ part_o,
                                                         const float *__restrict__ part_ml, OutT *o,
                                                         int ldo, int nq, int nkv, int hd) {
  const AttnGroup gr = groups[blockIdx.y];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int qloc = blockIdx.x * 4 + wave;
  const int G = nq / nkv;
  if (qloc >= gr.nq) return;
  const int tok_off = reqs[gr.req].tok_off;   // issued now, used for the store
  const int qrow = gr.q0 + qloc;
  const int qt = qrow / G, qg = gr.kvh * G + qrow % G;
  // Partials are read CH slots at a time, every load of a batch in flight
  // together; they are combined in slot order, as one slot at a time would.
  constexpr int CH = 8;
  constexpr int kMaxE = 256 / 64;             // head-dim elements per lane (head_dim <= 256)
  const float2 *ml = reinterpret_cast<const float2 *>(part_ml);
  float mx = -INFINITY;
  for (int c0 = 0; c0 < gr.n; c0 += CH) {
    float m[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c)
      m[c] = c0 + c < gr.n ? ml[(size_t)(gr.first_slot + c0 + c) * kAttnQB + qloc].x : -INFINITY;
#pragma unroll
    for (int c = 0; c < CH; ++c) mx = fmaxf(mx, m[c]);
  }
  float L = 0.f;
  float acc[kMaxE];
#pragma unroll
  for (int j = 0; j < kMaxE; ++j) acc[j] = 0.f;
  for (int c0 = 0; c0 < gr.n; c0 += CH) {
    float2 p[CH];
    float ov[CH][kMaxE];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const size_t base = (size_t)(gr.first_slot + c0 + c) * kAttnQB + qloc;
      const bool live = c0 + c < gr.n;
      p[c] = live ? ml[base] : make_float2(0.f, 0.f);
#pragma unroll
      for (int j = 0; j < kMaxE; ++j) ov[c][j] = live && lane + 64 * j < hd ? part_o[base * hd + lane + 64 * j] : 0.f;
    }
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      if (c0 + c >= gr.n) break;
      const float wgt = exp2f(p[c].x - mx);
      L += wgt * p[c].y;
#pragma unroll
      for (int j = 0; j < kMaxE; ++j) acc[j] += wgt * ov[c][j];
    }
  }
  const float inv = 1.0f / L;
  OutT *op = o + (size_t)(tok_off + qt) * ldo + (size_t)qg * hd;
#pragma unroll
  for (int j = 0; j < kMaxE; ++j)
    if (lane + 64 * j < hd) op[lane + 64 * j] = from_f32<OutT>(acc[j] * inv);
}

hipError_t launch_attention(const AttnArgs &a, bool bf16_mode, hipStream_t s) {
  if (a.n_items <= 0) return hipSuccess;
  if (bf16_mode) {
    if (a.n_blocks <= 0) return hipSuccess;
    dim3 grid(a.n_blocks);
    switch (a.hd) {
      case 32: hipLaunchKernelGGL((attention_bf16_kernel<32, attn_groups_per_wave(32)>), grid, dim3(256), 0, s, a); break;
      case 64: hipLaunchKernelGGL((attention_bf16_kernel<64, attn_groups_per_wave(64)>), grid, dim3(256), 0, s, a); break;
      case 128: hipLaunchKernelGGL((attention_bf16_kernel<128, attn_groups_per_wave(128)>), grid, dim3(256), 0, s, a); break;
      case 256: hipLaunchKernelGGL((attention_bf16_kernel<256, attn_groups_per_wave(256)>), grid, dim3(256), 0, s, a); break;
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
                             const float *part_o, const float *part_ml, void *o, int ldo, int nq,
                             int nkv, int hd, bool bf16_mode, hipStream_t s) {
  if (n_groups <= 0) return hipSuccess;
  if (hd > 256) return hipErrorInvalidValue;   // a lane holds at most 4 head-dim elements
  dim3 grid(kAttnQB / 4, n_groups);
  if (bf16_mode)
    hipLaunchKernelGGL(attn_merge_kernel<bf16>, grid, dim3(256), 0, s, groups, reqs, part_o, part_ml,
                       (bf16 *)o, ldo, nq, nkv, hd);
  else
    hipLaunchKernelGGL(attn_merge_kernel<float>, grid, dim3(256), 0, s, groups, reqs, part_o, part_ml,
                       (float *)o, ldo, nq, nkv, hd);
  return hipGetLastError();
}

}  // namespace rosa
