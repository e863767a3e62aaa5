// Ragged prefix + action attention of one layer.
//
// Request r's H_r action tokens (G = n_q / n_kv query heads per KV head, so
// G*H_r query rows per KV head) attend to its own key sequence: the P_r cached
// prefix keys of this layer followed by its H_r action keys; no other request
// and no padding is visible.  Scale 1/sqrt(head_dim); no causal mask.
//
// bf16 kernel (gfx950 MFMA).  A work item is (request, KV head, up to 128 NG
// query rows, key range).  Its four waves stream the key range through LDS in
// 32-key stages (K and V tiles; three stages in flight while one is used,
// copied by global_load_lds_dwordx4).  Each wave owns NG groups of 32 query
// rows (groups w and w + 4 of the item), so every K and V fragment it reads
// from LDS feeds the MFMAs of all its groups; NG is 2 where Q^T and O^T of two
// groups fit the register file (head_dim <= 128) and 1 otherwise.
// Per 32-key tile a wave computes S^T = K Q^T with v_mfma_f32_32x32x16_bf16
// (K from LDS, Q^T held in registers for the whole item), so that each lane
// owns one query column: the online-softmax max and sum are in-lane plus one
// exchange between the two 32-lane halves, and rescaling the output is
// per-lane.  O^T += V^T P^T then takes P^T straight from the S^T registers
// (the contraction's key order is permuted identically on both operands) and
// V^T from the row-major V tile with the LDS transpose read
// ds_read_b64_tr_b16, so the tile is stored as it streams in.
// Work items that cover part of a request's keys write unnormalized partial
// results that a merge kernel combines in a fixed order.
#include <math.h>

#include "rosa_device.h"
#include "rosa_internal.h"

namespace rosa {

namespace at {
constexpr int TK = 32;   // keys per LDS stage
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
// Chunk swizzle of LDS rows: 16-byte chunk c of row r is stored at c ^ swz(r),
// swz(r) = the two 2-bit halves of r % 16 swapped.  The 16 consecutive rows
// that one 16-lane group reads at one chunk (K operand), and the 4 rows x 4
// chunks that the transpose reads of a 32-lane half touch (V operand), then
// fall in distinct bank groups.
__device__ __forceinline__ int swz(int r, int cpr) { return (((r & 3) << 2) | ((r >> 2) & 3)) & (cpr - 1); }
}  // namespace at

#define ROSA_LDS_A(p) ((__attribute__((address_space(3))) void *)(p))

__device__ __forceinline__ bf16x8 lds_tr_pair(const uint8_t *p0, const uint8_t *p1) {
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

// Maps block b to a work item so that the items of one request (consecutive
// in the list) run on the same XCD at about the same time and share its L2:
// blocks are handed to the 8 XCDs round-robin, and XCD x takes the x-th
// eighth of the list in order.
__device__ __forceinline__ int xcd_item(int b, int n_items) {
  const int x = b & 7, q = b >> 3;
  const int per = n_items >> 3, extra = n_items & 7;
  const int start = x * per + min(x, extra);
  const int len = per + (x < extra ? 1 : 0);
  return q < len ? start + q : -1;
}

template <int HD, int NG>
__global__ void __launch_bounds__(256, 1) attention_bf16_kernel(AttnArgs a) {
  using at::TK;
  using T = AttnTile<HD>;
  constexpr int NS = HD / 16;   // MFMA k-steps over head_dim for S
  constexpr int NT = HD / 32;   // 32-row output tiles over head_dim
  constexpr int CPR = T::CPR, ROWB = T::ROWB, TILEB = T::TILEB;
  // Four LDS stages (K tile, then V tile): three tiles are in flight while
  // one is used.  Each stage is its own LDS object, so the compiler's own
  // waits never cover the copies of later stages.
  __shared__ __attribute__((aligned(1024))) uint8_t S0[2 * TILEB];
  __shared__ __attribute__((aligned(1024))) uint8_t S1[2 * TILEB];
  __shared__ __attribute__((aligned(1024))) uint8_t S2[2 * TILEB];
  __shared__ __attribute__((aligned(1024))) uint8_t S3[2 * TILEB];

  const int item = xcd_item(blockIdx.x, a.n_items);
  if (item < 0) return;
  const AttnItem it = a.items[item];
  const ReqDesc rq = a.reqs[it.req];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6) & 3;   // wave-uniform, in an SGPR
  const int half = lane >> 5;
  const int G = a.nq / a.nkv;
  const bf16 *qkv = reinterpret_cast<const bf16 *>(a.qkv);

  // Q^T operand of group g, held for the whole item: lane holds
  // Q[row][16 s + 8 half .. + 7] for its row; rows past the item's queries
  // read the item's first row instead (their results are never stored).
  bf16x8 qf[NG][NS];
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int loc = 32 * (wave + 4 * g) + (lane & 31);
    const int qrow = it.q0 + (loc < it.nq ? loc : 0);
    const bf16 *qp = qkv + (size_t)(rq.tok_off + qrow / G) * a.ldqkv + (size_t)(it.kvh * G + qrow % G) * HD + half * 8;
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[g][s] = *reinterpret_cast<const bf16x8 *>(qp + 16 * s);
  }

  const size_t prow = (size_t)a.nkv * HD;   // prefix row stride (elements)
  const bf16 *pk = reinterpret_cast<const bf16 *>(rq.pk) + (size_t)a.layer * rq.P * prow + (size_t)it.kvh * HD;
  const bf16 *pv = reinterpret_cast<const bf16 *>(rq.pv) + (size_t)a.layer * rq.P * prow + (size_t)it.kvh * HD;
  const bf16 *ak = qkv + (size_t)rq.tok_off * a.ldqkv + (size_t)(a.nq + it.kvh) * HD;
  const bf16 *av = qkv + (size_t)rq.tok_off * a.ldqkv + (size_t)(a.nq + a.nkv + it.kvh) * HD;
  const long ldq = a.ldqkv;

  // Copies: 1 KB units, unit u of the K tile (then of the V tile) by wave
  // u % 4; lane i fills physical chunk i % CPR of row u * RPU + i / CPR, which
  // holds logical chunk (i % CPR) ^ swz(row).  Keys past the range load the
  // last valid key (finite values; their scores are masked).
  // Tiles that lie wholly in the prefix (all but at most two per item) take
  // their sources from a uniform base plus per-lane offsets fixed for the whole
  // item; the others compute each lane's key.  Only the addresses depend on
  // the case: the copies themselves are issued after the join, so the
  // compiler's tracking of the pending LDS writes stays exact (a copy issued
  // inside a branch makes it wait for every copy before the next LDS read).
  constexpr int UPW = (T::UNITS / 2 + 3) / 4;    // K (or V) units per copying wave
  int poff[UPW];
#pragma unroll
  for (int j = 0; j < UPW; ++j) {
    const int row = (4 * j + wave) * T::RPU + lane / CPR;
    poff[j] = row * (int)prow + (((lane % CPR) ^ at::swz(row, CPR)) << 3);
  }
  auto issue = [&](uint8_t *st, int kt0) {
    const bf16 *ksrc[UPW], *vsrc[UPW];
    if (kt0 + TK <= rq.P && kt0 + TK <= it.kend) {
      const bf16 *kb = pk + (size_t)kt0 * prow;
      const bf16 *vb = pv + (size_t)kt0 * prow;
#pragma unroll
      for (int j = 0; j < UPW; ++j) { ksrc[j] = kb + poff[j]; vsrc[j] = vb + poff[j]; }
    } else {
#pragma unroll
      for (int j = 0; j < UPW; ++j) {
        const int row = (4 * j + wave) * T::RPU + lane / CPR;
        const int c = (lane % CPR) ^ at::swz(row, CPR);
        const int key = min(kt0 + row, it.kend - 1);
        const bool pre = key < rq.P;
        const long roff = (pre ? (long)key * (long)prow : (long)(key - rq.P) * ldq) + c * 8;
        ksrc[j] = (pre ? pk : ak) + roff;
        vsrc[j] = (pre ? pv : av) + roff;
      }
    }
#pragma unroll
    for (int j = 0; j < UPW; ++j)
      if (4 * j + wave < T::UNITS / 2)
        __builtin_amdgcn_global_load_lds((const void *)ksrc[j], ROSA_LDS_A(st + (4 * j + wave) * 1024), 16, 0, 0);
#pragma unroll
    for (int j = 0; j < UPW; ++j)
      if (4 * j + wave < T::UNITS / 2)
        __builtin_amdgcn_global_load_lds((const void *)vsrc[j], ROSA_LDS_A(st + TILEB + (4 * j + wave) * 1024), 16, 0, 0);
  };

  f32x16 o[NG][NT];
  // Softmax without rescaling the output inside the key loop: each query's
  // reference max m_ref is its max over the item's first 32-key tile, and
  // P = 2^((s - m_ref) log2(e) / sqrt(hd)) may exceed 1.  The loop tracks the
  // true max; if any query's later scores exceed its reference by more than
  // 2^64 (room to spare below fp32 overflow for the sums), the block runs the
  // item a second time with the true max as reference, where P <= 1.  Either
  // way the output accumulators are only touched by MFMAs in the loop.
  float m_ref[NG], m_true[NG], l_run[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) m_true[g] = -INFINITY;
  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);   // log2(e) / sqrt(hd)
  const float over = 64.0f / sl2;           // raw score excess that asks for the second pass

  // K operand: row lane%32, logical chunk 2 ks + half.
  const int krow = lane & 31;
  const int kbase = krow * ROWB;
  const int ksw = at::swz(krow, CPR);
  // V transpose reads: source lane s of 16-lane group G16 reads 8 bytes at
  // row 16 ks + 4 half + s/4 (and 8 rows further), head-dim column
  // 32 n + 16 G16 + 4 (s%4).
  const int src16 = lane & 15, g16 = (lane >> 4) & 1;
  const int vcol = 16 * g16 + 4 * (src16 & 3);

  const int nkt = (it.kend - it.kbeg + TK - 1) / TK;
  auto issue_t = [&](uint8_t *st, int t) { issue(st, it.kbeg + min(t, nkt - 1) * TK); };

  // A wave's groups past the item's rows compute on a clamped row (each wave
  // has its own SIMD; the results are never stored).
  int ovf = 0;
  auto tile = [&](const uint8_t *st, int kt0, bool first, bool pass0) {
    // S^T (32 keys x 32 queries) per group: lane holds query lane%32;
    // register r holds key kt0 + (r/4)*8 + 4 half + r%4.
    f32x16 s[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[g][r] = 0.f;
#pragma unroll
    for (int ks = 0; ks < NS; ++ks) {
      const bf16x8 kf = *reinterpret_cast<const bf16x8 *>(st + kbase + (((2 * ks + half) ^ ksw) << 4));
#pragma unroll
      for (int g = 0; g < NG; ++g) s[g] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[g][ks], s[g], 0, 0, 0);
    }
    // Keep about two K fragments in flight: one LDS read, then the MFMAs
    // that use it (the register file holds Q^T and O^T).
#pragma unroll
    for (int ks = 0; ks < NS; ++ks) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, NG, 0);
    }
    bf16x8 pf[NG][2];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      if (kt0 + TK > it.kend) {               // last, partial tile
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kt0 + (r >> 2) * 8 + half * 4 + (r & 3);
          if (key >= it.kend) s[g][r] = -INFINITY;
        }
      }
      float tmax = s[g][0];
#pragma unroll
      for (int r = 1; r < 16; ++r) tmax = fmaxf(tmax, s[g][r]);
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
      if (first && pass0) m_ref[g] = tmax;
      m_true[g] = fmaxf(m_true[g], tmax);
      ovf |= tmax > m_ref[g] + over;
      const float mb = -m_ref[g] * sl2;
      float psum = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float pe = __builtin_amdgcn_exp2f(fmaf(s[g][r], sl2, mb));
        psum += pe;
        pf[g][r >> 3][r & 7] = (bf16)pe;
      }
      psum += __shfl_xor(psum, 32, 64);
      l_run[g] += psum;
    }
    // O^T (head_dim x queries) += V^T P^T; k-step ks uses P^T registers
    // 8 ks .. 8 ks + 7, i.e. keys 16 ks + 8 (i/4) + 4 half + i%4.
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int r0 = ks * 16 + half * 4 + (src16 >> 2);
      const uint8_t *v0 = st + TILEB + r0 * ROWB;
      const uint8_t *v1 = st + TILEB + (r0 + 8) * ROWB;
      const int sw0 = at::swz(r0, CPR), sw1 = at::swz(r0 + 8, CPR);
#pragma unroll
      for (int n = 0; n < NT; ++n) {
        const int x = n * 32 + vcol;   // head-dim column (bf16 index)
        const int off0 = (((x >> 3) ^ sw0) << 4) + ((x & 7) << 1);
        const int off1 = (((x >> 3) ^ sw1) << 4) + ((x & 7) << 1);
        const bf16x8 vf = lds_tr_pair(v0 + off0, v1 + off1);
#pragma unroll
        for (int g = 0; g < NG; ++g) o[g][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[g][ks], o[g][n], 0, 0, 0);
      }
    }
#pragma unroll
    for (int n = 0; n < 2 * NT; ++n) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 1);
      __builtin_amdgcn_sched_group_barrier(0x008, NG, 1);
    }
  };
  // Ring of four stages; tile t lives in stage t % 4.  Copies past the last
  // tile repeat it (harmless), so every step issues exactly one stage and the
  // wait count stays uniform.
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
    auto step = [&](uint8_t *cur, uint8_t *refill, int t) {
      __builtin_amdgcn_s_waitcnt(T::WAIT);    // this wave's copies of tile t have landed
      __builtin_amdgcn_s_barrier();           // ... and every wave's; tile t-1's stage is free
      __builtin_amdgcn_sched_barrier(0);
      issue_t(refill, t + 3);
      tile(cur, it.kbeg + t * TK, t == 0, pass0);
    };
    issue_t(S0, 0);
    issue_t(S1, 1);
    issue_t(S2, 2);
    // Whole groups of four tiles without branches between the steps (a join
    // would make the compiler wait for every pending copy before the next LDS
    // read), then the last one to three tiles.
    int t = 0;
    for (; t + 4 <= nkt; t += 4) {
      step(S0, S3, t);
      step(S1, S0, t + 1);
      step(S2, S1, t + 2);
      step(S3, S2, t + 3);
    }
    if (t < nkt) {
      step(S0, S3, t);
      if (t + 1 < nkt) {
        step(S1, S0, t + 1);
        if (t + 2 < nkt) step(S2, S1, t + 2);
      }
    }
    __builtin_amdgcn_s_waitcnt(T::WAIT0);   // no copy may outlive the pass (or the block's LDS)
    // Block-uniform decision: every wave has finished reading the stages.
    if (!pass0 || !__syncthreads_or(ovf)) break;
#pragma unroll
    for (int g = 0; g < NG; ++g) m_ref[g] = m_true[g];
  }

  // Accumulator layout: lane holds query (lane & 31) of the group; register r
  // of tile n holds head-dim index 32 n + (r/4)*8 + 4 half + r%4.
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int loc = 32 * (wave + 4 * g) + (lane & 31);
    if (loc >= it.nq) continue;
    if (it.slot < 0) {
      const int qrow = it.q0 + loc;
      const float inv = 1.0f / l_run[g];
      bf16 *op = reinterpret_cast<bf16 *>(a.o) + (size_t)(rq.tok_off + qrow / G) * a.ldo +
                 (size_t)(it.kvh * G + qrow % G) * HD;
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          bf16x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = (bf16)(o[g][n][rg * 4 + e] * inv);
          *reinterpret_cast<bf16x4 *>(op + n * 32 + rg * 8 + half * 4) = v;
        }
    } else {
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
        pm[1] = l_run[g];
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
  const ReqDesc rq = reqs[gr.req];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int qloc = blockIdx.x * 4 + wave;
  const int G = nq / nkv;
  if (qloc >= gr.nq) return;
  const int qrow = gr.q0 + qloc;
  const int qt = qrow / G, qg = gr.kvh * G + qrow % G;
  float mx = -INFINITY;
  for (int c = 0; c < gr.n; ++c) mx = fmaxf(mx, part_ml[((size_t)(gr.first_slot + c) * kAttnQB + qloc) * 2]);
  float L = 0.f;
  for (int c = 0; c < gr.n; ++c) {
    const float *pm = part_ml + ((size_t)(gr.first_slot + c) * kAttnQB + qloc) * 2;
    L += exp2f(pm[0] - mx) * pm[1];
  }
  const float inv = 1.0f / L;
  OutT *op = o + (size_t)(rq.tok_off + qt) * ldo + (size_t)qg * hd;
  for (int e = lane; e < hd; e += 64) {
    float acc = 0.f;
    for (int c = 0; c < gr.n; ++c) {
      const size_t base = (size_t)(gr.first_slot + c) * kAttnQB + qloc;
      acc += exp2f(part_ml[base * 2] - mx) * part_o[base * hd + e];
    }
    op[e] = from_f32<OutT>(acc * inv);
  }
}

hipError_t launch_attention(const AttnArgs &a, bool bf16_mode, hipStream_t s) {
  if (a.n_items <= 0) return hipSuccess;
  if (bf16_mode) {
    dim3 grid((a.n_items + 7) / 8 * 8);
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
