// Ragged prefix + action attention of one layer.
//
// Request r's H_r action tokens (G = n_q / n_kv query heads per KV head, so
// G*H_r query rows per KV head) attend to its own key sequence: the P_r cached
// prefix keys of this layer followed by its H_r action keys; no other request
// and no padding is visible.  Scale 1/sqrt(head_dim); no causal mask.
//
// bf16 kernel (gfx950 MFMA).  A work item is (request, KV head, block of 128
// query rows, key range).  Its four waves own 32 query rows each and stream the
// key range through LDS in 64-key tiles (K and V tiles double-buffered; the
// next tile's global loads are in flight while the current one is consumed).
// Per 64-key tile a wave computes S^T = K Q^T with v_mfma_f32_32x32x16_bf16
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
constexpr int TK = 64;   // keys per LDS tile
}

__device__ __forceinline__ bf16x8 lds_tr_pair(const bf16 *p0, const bf16 *p1) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  const i16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(p0));
  const i16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(p1));
  const uint2 u0 = __builtin_bit_cast(uint2, v0);
  const uint2 u1 = __builtin_bit_cast(uint2, v1);
  return __builtin_bit_cast(bf16x8, make_uint4(u0.x, u0.y, u1.x, u1.y));
}

template <int HD>
__global__ void __launch_bounds__(256) attention_bf16_kernel(AttnArgs a) {
  using at::TK;
  constexpr int KW = HD + 8;    // K tile row stride (bf16): 16-byte pad
  constexpr int VW = HD + 32;   // V tile row stride (bf16): 64-byte pad
  constexpr int NS = HD / 16;   // MFMA k-steps over head_dim for S
  constexpr int NT = HD / 32;   // 32-row output tiles over head_dim
  constexpr int CPR = HD / 8;   // 16-byte chunks per K/V row
  constexpr int CPT = TK * CPR / 256;
  static_assert(CPT >= 1, "head_dim too small");
  __shared__ __attribute__((aligned(16))) bf16 Ks[2][TK * KW];
  __shared__ __attribute__((aligned(16))) bf16 Vs[2][TK * VW];

  const AttnItem it = a.items[blockIdx.x];
  const ReqDesc rq = a.reqs[it.req];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int half = lane >> 5;
  const int G = a.nq / a.nkv;
  const int nrows = rq.H * G;
  const int qloc = wave * 32 + (lane & 31);
  const int qrow = it.qb * kAttnQB + qloc;
  const bool qvalid = qrow < nrows;
  const int qt = qvalid ? qrow / G : 0;
  const int qg = it.kvh * G + (qvalid ? qrow % G : 0);
  const bf16 *qkv = reinterpret_cast<const bf16 *>(a.qkv);

  // Q^T operand: lane holds Q[qrow][16 s + 8 half .. + 7] for k-step s.
  bf16x8 qf[NS];
  {
    const bf16 *qp = qkv + (size_t)(rq.tok_off + qt) * a.ldqkv + (size_t)qg * HD + half * 8;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const uint4 v = qvalid ? *reinterpret_cast<const uint4 *>(qp + 16 * s) : make_uint4(0, 0, 0, 0);
      qf[s] = __builtin_bit_cast(bf16x8, v);
    }
  }

  const size_t prow = (size_t)a.nkv * HD;   // prefix row stride (elements)
  const bf16 *pk = reinterpret_cast<const bf16 *>(rq.pk) + (size_t)a.layer * rq.P * prow + (size_t)it.kvh * HD;
  const bf16 *pv = reinterpret_cast<const bf16 *>(rq.pv) + (size_t)a.layer * rq.P * prow + (size_t)it.kvh * HD;
  const bf16 *ak = qkv + (size_t)rq.tok_off * a.ldqkv + (size_t)(a.nq + it.kvh) * HD;
  const bf16 *av = qkv + (size_t)rq.tok_off * a.ldqkv + (size_t)(a.nq + a.nkv + it.kvh) * HD;

  uint4 rk[CPT], rv[CPT];
  auto load_tile = [&](int kt0) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + 256 * i, row = c / CPR, c8 = (c % CPR) * 8;
      const int key = kt0 + row;
      if (key < it.kend) {
        const bf16 *sk = key < rq.P ? pk + (size_t)key * prow : ak + (size_t)(key - rq.P) * a.ldqkv;
        const bf16 *sv = key < rq.P ? pv + (size_t)key * prow : av + (size_t)(key - rq.P) * a.ldqkv;
        rk[i] = *reinterpret_cast<const uint4 *>(sk + c8);
        rv[i] = *reinterpret_cast<const uint4 *>(sv + c8);
      } else {
        rk[i] = make_uint4(0, 0, 0, 0);
        rv[i] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = tid + 256 * i, row = c / CPR, c8 = (c % CPR) * 8;
      *reinterpret_cast<uint4 *>(&Ks[buf][row * KW + c8]) = rk[i];
      *reinterpret_cast<uint4 *>(&Vs[buf][row * VW + c8]) = rv[i];
    }
  };

  f32x16 o[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[n][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);   // log2(e) / sqrt(hd)

  const int nkt = (it.kend - it.kbeg + TK - 1) / TK;
  load_tile(it.kbeg);
  store_tile(0);
  __syncthreads();
  for (int t = 0; t < nkt; ++t) {
    const int cur = t & 1;
    const int kt0 = it.kbeg + t * TK;
    if (t + 1 < nkt) load_tile(kt0 + TK);

    // S^T (keys x queries) for two 32-key sub-tiles.
    f32x16 s[2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[sub][r] = 0.f;
      const bf16 *kb = &Ks[cur][(sub * 32 + (lane & 31)) * KW + half * 8];
#pragma unroll
      for (int ks = 0; ks < NS; ++ks) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8 *>(kb + ks * 16);
        s[sub] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[sub], 0, 0, 0);
      }
    }
    // Lane holds query (lane & 31); register r of sub-tile `sub` holds key
    // kt0 + 32 sub + (r/4)*8 + 4 half + r%4.
    float tmax = -INFINITY;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kt0 + sub * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
        const float v = key < it.kend ? s[sub][r] * sl2 : -INFINITY;
        s[sub][r] = v;
        tmax = fmaxf(tmax, v);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float m_new = fmaxf(m_run, tmax);     // finite: every tile has a valid key
    const float alpha = exp2f(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = exp2f(s[sub][r] - m_new);
        s[sub][r] = p;
        psum += p;
      }
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[n][r] *= alpha;

    // P^T operands: k-step ks of sub-tile sub uses registers 8 ks .. 8 ks + 7,
    // i.e. keys 16 ks + 8 (i/4) + 4 half + i%4 for element i.
    bf16x8 pf[2][2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int i = 0; i < 8; ++i) pf[sub][ks][i] = (bf16)s[sub][8 * ks + i];

    // O^T (head_dim x queries) += V^T P^T.  The V^T operand of lane l needs
    // V[key(i)][32 n + l%32]; each transpose read delivers four consecutive keys.
    const int src = lane & 15;
    const int mcol = 16 * ((lane >> 4) & 1) + 4 * (src & 3);
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int krow = sub * 32 + ks * 16 + half * 4 + (src >> 2);
        const bf16 *vb = &Vs[cur][krow * VW + mcol];
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          const bf16x8 vf = lds_tr_pair(vb + n * 32, vb + 8 * VW + n * 32);
          o[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[sub][ks], o[n], 0, 0, 0);
        }
      }

    if (t + 1 < nkt) store_tile(cur ^ 1);
    __syncthreads();
  }

  // Accumulator layout: lane holds query (lane & 31); register r of tile n holds
  // head-dim index 32 n + (r/4)*8 + 4 half + r%4.
  if (it.slot < 0) {
    if (!qvalid) return;
    const float inv = 1.0f / l_run;
    bf16 *op = reinterpret_cast<bf16 *>(a.o) + (size_t)(rq.tok_off + qt) * a.ldo + (size_t)qg * HD;
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        bf16x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (bf16)(o[n][rg * 4 + e] * inv);
        *reinterpret_cast<bf16x4 *>(op + n * 32 + rg * 8 + half * 4) = v;
      }
  } else {
    float *po = a.part_o + ((size_t)it.slot * kAttnQB + qloc) * HD;
#pragma unroll
    for (int n = 0; n < NT; ++n)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const float4 v = make_float4(o[n][rg * 4 + 0], o[n][rg * 4 + 1], o[n][rg * 4 + 2], o[n][rg * 4 + 3]);
        *reinterpret_cast<float4 *>(po + n * 32 + rg * 8 + half * 4) = v;
      }
    if (half == 0) {
      float *pm = a.part_ml + ((size_t)it.slot * kAttnQB + qloc) * 2;
      pm[0] = m_run;
      pm[1] = l_run;
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
  const int qrow = it.qb * kAttnQB + blockIdx.y * 4 + wave;
  if (qrow >= rq.H * G) return;
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
  const int qrow = gr.qb * kAttnQB + qloc;
  if (qrow >= rq.H * G) return;
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
    dim3 grid(a.n_items);
    switch (a.hd) {
      case 32: hipLaunchKernelGGL(attention_bf16_kernel<32>, grid, dim3(256), 0, s, a); break;
      case 64: hipLaunchKernelGGL(attention_bf16_kernel<64>, grid, dim3(256), 0, s, a); break;
      case 128: hipLaunchKernelGGL(attention_bf16_kernel<128>, grid, dim3(256), 0, s, a); break;
      case 256: hipLaunchKernelGGL(attention_bf16_kernel<256>, grid, dim3(256), 0, s, a); break;
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
