// C ABI of the rosa library: handle lifetime, validation, the batch plan and
// the step loop that enqueues the kernels on the handle's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <thread>
#include <queue>
#include <vector>

#include "../../include/rosa.h"
#include "../../include/rosa_debug.h"
#include "rosa_internal.h"

using namespace rosa;

// Most rows a lane-step may have for its unsplit output projection and
// MLP-down to defer their norms to the next product.  Above it a separate
// norm launch costs less than the completing products' longer epilogues.
constexpr int kDeferMaxRows = 1024;

// Attention launch order.  The kernel's blocks are persistent: block b runs
// the items of its own list one after another, and blocks reach the 8 XCDs
// round-robin (block b on XCD b % 8).  Two levels of longest-processing-time
// packing (largest first onto the least loaded), so the blocks finish
// together:
//   - onto XCDs: a request's items go to one XCD as a unit (its query blocks
//     read the same keys through that XCD's L2); a request holding more than
//     1/16 of the launch's work goes item by item instead;
//   - on each XCD: its items onto its blocks, one block per item while the
//     busiest XCD has no more items than kAttnBlocks / 8.
// Item cost = 32-key steps + a fixed overhead.  Appends the block lists to
// out (item index per entry) and next (the index, relative to this table, of
// the same block's next entry, -1 after its last): entries 0 .. n_blocks-1
// are the blocks' first items (-1: an idle block), the others follow block
// by block.  Returns n_blocks.  The order never changes what an item computes.
namespace rosa {
int attn_launch_order(const std::vector<AttnItem> &items, const std::vector<std::pair<int, int>> &ranges,
                      std::vector<int32_t> &out, std::vector<int32_t> &next) {
  constexpr int64_t kItemOverheadSteps = 6;   // fixed cost of an item in a persistent block, in 32-key steps
  auto icost = [&](int it) -> int64_t { return (items[it].kend - items[it].kbeg + 31) / 32 + kItemOverheadSteps; };
  struct Unit { int lo, hi; int64_t cost; };   // items [lo, hi) placed together
  int64_t total = 0;
  for (const auto &r : ranges)
    for (int j = r.first; j < r.second; ++j) total += icost(j);
  std::vector<Unit> units;
  for (const auto &r : ranges) {
    int64_t c = 0;
    for (int j = r.first; j < r.second; ++j) c += icost(j);
    if (16 * c > total) {
      for (int j = r.first; j < r.second; ++j) units.push_back({j, j + 1, icost(j)});
    } else {
      units.push_back({r.first, r.second, c});
    }
  }
  std::stable_sort(units.begin(), units.end(), [](const Unit &a, const Unit &b2) { return a.cost > b2.cost; });
  int64_t xload[8] = {};
  std::vector<std::vector<int>> xitems(8);
  for (const Unit &u : units) {
    int best = 0;
    for (int x = 1; x < 8; ++x)
      if (xload[x] < xload[best]) best = x;
    xload[best] += u.cost;
    for (int it = u.lo; it < u.hi; ++it) xitems[best].push_back(it);
  }
  size_t most = 1;
  for (int x = 0; x < 8; ++x) most = std::max(most, xitems[x].size());
  const int per_x = std::min(kAttnBlocks / 8, (int)most);
  const int nb = 8 * per_x;
  std::vector<std::vector<int>> bins(nb);
  using LB = std::pair<int64_t, int>;       // (load, bin) min-heap per XCD
  for (int x = 0; x < 8; ++x) {
    std::stable_sort(xitems[x].begin(), xitems[x].end(), [&](int a, int b2) { return icost(a) > icost(b2); });
    std::priority_queue<LB, std::vector<LB>, std::greater<LB>> heap;
    for (int j = 0; j < per_x; ++j) heap.push({0, j});
    for (int it : xitems[x]) {
      LB lb = heap.top();
      heap.pop();
      bins[x + 8 * lb.second].push_back(it);
      lb.first += icost(it);
      heap.push(lb);
    }
  }
  const size_t at = out.size();
  out.resize(at + nb, -1);
  next.resize(at + nb, -1);
  for (int b = 0; b < nb; ++b) {
    if (bins[b].empty()) continue;
    out[at + b] = bins[b][0];
    int32_t prev = b;                       // relative index of the entry to link from
    for (size_t q = 1; q < bins[b].size(); ++q) {
      const int32_t e = (int32_t)(out.size() - at);
      out.push_back(bins[b][q]);
      next.push_back(-1);
      next[at + prev] = e;
      prev = e;
    }
  }
  return nb;
}

void attn_order_items(const std::vector<AttnItem> &items, const int32_t *order, const int32_t *next, size_t n,
                      AttnItem *dst) {
  for (size_t e = 0; e < n; ++e) {
    if (order[e] >= 0) {
      dst[e] = items[order[e]];
    } else {
      dst[e] = AttnItem{};
      dst[e].nq = 0;
    }
    dst[e].next = next[e];
  }
}

uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

hipError_t upload_weights_kb32(void *dst, const float *src, int L, int K, int N) {
  const size_t per = (size_t)K * N;
  std::vector<uint16_t> tmp(per * L);
  auto work = [&](int l) {
    const float *s = src + per * l;
    uint16_t *d = tmp.data() + per * l;
    for (int k = 0; k < K; ++k)
      for (int n = 0; n < N; ++n) d[kb32_offset(N, n, k)] = f32_to_bf16_rne(s[(size_t)k * N + n]);
  };
  std::vector<std::thread> th;
  const int nt = std::max(1, std::min(L, 8));
  for (int t = 0; t < nt; ++t)
    th.emplace_back([&, t] { for (int l = t; l < L; l += nt) work(l); });
  for (auto &x : th) x.join();
  return hipMemcpy(dst, tmp.data(), tmp.size() * 2, hipMemcpyHostToDevice);
}

hipError_t upload_weights_transposed(void *dst, const float *src, int L, int K, int N, bool bf16) {
  const size_t per = (size_t)K * N;
  std::vector<uint8_t> tmp(per * L * (bf16 ? 2 : 4));
  auto work = [&](int l) {
    const float *s = src + per * l;
    for (int k0 = 0; k0 < K; k0 += 64)
      for (int n0 = 0; n0 < N; n0 += 64)
        for (int n = n0; n < std::min(N, n0 + 64); ++n)
          for (int k = k0; k < std::min(K, k0 + 64); ++k) {
            const float v = s[(size_t)k * N + n];
            const size_t di = per * l + (size_t)n * K + k;
            if (bf16) reinterpret_cast<uint16_t *>(tmp.data())[di] = f32_to_bf16_rne(v);
            else reinterpret_cast<float *>(tmp.data())[di] = v;
          }
  };
  std::vector<std::thread> th;
  const int nt = std::max(1, std::min(L, 8));
  for (int t = 0; t < nt; ++t)
    th.emplace_back([&, t] { for (int l = t; l < L; l += nt) work(l); });
  for (auto &x : th) x.join();
  return hipMemcpy(dst, tmp.data(), tmp.size(), hipMemcpyHostToDevice);
}
}  // namespace rosa

namespace {

constexpr int kSplitTarget = kAttnSplitTarget;
constexpr int kMinSplitKeys = kAttnMinSplitKeys;
constexpr int kMaxSlots = kAttnMaxSlots;
constexpr int kMaxLanes = 4;
constexpr int kMinLaneRequests = 64;  // a batch splits into lanes only with at least this many requests per lane

enum KernelClass {
  kcTime = 0, kcSetup, kcInProj, kcModNorm, kcGemmQKV, kcAttention, kcMerge, kcGemmO, kcGemmUp,
  kcGemmDown, kcFinal, kcCount
};
const char *kClassNames[kcCount] = {"time_conditioning", "setup_rows", "in_proj", "modnorm", "gemm_qkv",
                                    "attention", "attn_merge", "gemm_o", "gemm_up", "gemm_down",
                                    "final_euler"};

thread_local std::string g_create_error;

struct Plan {
  std::vector<int32_t> order;        // plan position -> caller index
  std::vector<int32_t> tok_off;      // by plan position
  std::vector<int32_t> steps;        // by plan position: Euler steps this call runs
  std::vector<int32_t> m_k;          // per step
  std::vector<int32_t> n_active;     // per step
  std::vector<float> taus;
  std::vector<int32_t> tau_idx;      // [max_K][n]
  // Attention work: set 0 serves joint (or, alternating, cross-attention)
  // layers, set 1 the self-attention layers of the alternating layout.  The
  // device holds set 0's items then set 1's (likewise groups); launch orders
  // index the whole item array; partial slots are numbered across both sets.
  struct AttnSet {
    std::vector<AttnItem> items;
    std::vector<AttnGroup> groups;
    std::vector<int32_t> items_upto;   // items of plan requests [0, r]
    std::vector<int32_t> groups_upto;
    int item_base = 0, group_base = 0;
  };
  AttnSet sets[2];
  int n_sets = 1;
  int slots = 0;
  int M0 = 0, Kmax = 0;
  // Lanes: disjoint request sets run as independent sub-batches on their own
  // streams.  Lane l owns plan positions [req_lo, req_hi) and stacked rows
  // [row_lo, row_hi); at step k its active requests and rows are the prefixes
  // n_act[k] and m[k] of those ranges (each lane is sorted by K descending).
  struct Lane {
    int req_lo = 0, req_hi = 0, row_lo = 0, row_hi = 0;
    std::vector<int32_t> n_act, m;
    // Per attention set and step: offset of the attention launch order in
    // attn_lists, and the launch's block count.
    std::vector<int32_t> list_at[2], list_blocks[2];
  };
  std::vector<Lane> lanes;
  // Attention launch orders, one per distinct set of active requests of a
  // lane: the persistent blocks' item lists (item index per entry, -1: an
  // idle block) and each entry's link to its block's next entry.
  std::vector<int32_t> attn_lists, attn_next;
};

}  // namespace

struct rosa_batch {
  rosa_model_config cfg{};
  rosa_capacity cap{};
  Dims dims{};
  bool bf16 = true;
  size_t esz = 2;
  int device = 0;
  hipStream_t stream = nullptr;
  bool poisoned = false;
  int gemm_cfg = -1;                 // forced projection block configuration, -1: cost model
  // bf16: u, o and g (the projections' A operands) are kb32 with planes of
  // kb_rows rows (the handle's row capacity); 0 in fp32 mode (row-major).
  int kb_rows = 0;
  // Lanes: sub-batches run concurrently; lane 0 uses `stream`, lane l > 0 its own
  // stream (default priority), forked after the time conditioning and joined back.
  int lanes = 1;
  hipStream_t lane_stream[kMaxLanes] = {};
  hipEvent_t ev_fork = nullptr, ev_join[kMaxLanes] = {};
  std::string last_error;

  // weights on the device
  float *w_in = nullptr, *b_in = nullptr, *b_t1 = nullptr, *b_t2 = nullptr, *b_modall = nullptr;
  float *w_out = nullptr, *b_out = nullptr;
  void *wt_out = nullptr;            // bf16 mode: W_out transposed, [A][d]
  void *w_t1 = nullptr, *w_t2 = nullptr, *w_modall = nullptr;       // [K][N], activation dtype
  void *wt_qkv = nullptr, *wt_o = nullptr, *wt_up = nullptr, *wt_down = nullptr;  // [L][N][K]

  // workspaces
  float *x = nullptr, *h = nullptr;
  void *u = nullptr, *qkv = nullptr, *o = nullptr, *g = nullptr;
  int32_t *row_req = nullptr, *rowmod = nullptr, *ident = nullptr;
  float *modtab = nullptr, *emb = nullptr, *tc1 = nullptr, *tc2 = nullptr, *gemv_ws = nullptr;
  float *part_o = nullptr, *part_ml = nullptr;
  float *gemm_part = nullptr;        // K-slice products of split projections (one lane only)
  size_t gemm_part_floats = 0;
  // bf16 deferred norms (unsplit output projection and MLP-down): per row the
  // sums of squares of h over its 32-column blocks, and the norms' shift
  // vectors multiplied by W_qkv and W_up, [L][modulation row][qkv_dim + dff].
  float *dn_ss = nullptr, *dn_shift = nullptr;
  int max_items = 0;                 // attention work items per call, both sets
  int max_slots = 0;                 // partial-result slots per call, both sets


  // plan buffers: device region + two pinned host staging copies
  void *d_plan = nullptr;
  void *h_plan[2] = {nullptr, nullptr};
  hipEvent_t plan_copied[2] = {nullptr, nullptr};
  bool plan_pending[2] = {false, false};
  int plan_flip = 0;
  size_t plan_bytes = 0;
  size_t off_reqs = 0, off_tau_idx = 0, off_taus = 0, off_items = 0, off_groups = 0, off_lists = 0;
  size_t max_list_ints = 0;

  std::vector<void *> allocations;

  // profiling
  bool prof = false;
  struct Pending { int cls; hipEvent_t a, b; };
  std::vector<Pending> pending;
  std::vector<hipEvent_t> free_events;
  int64_t prof_launches[kcCount] = {};
  double prof_ms[kcCount] = {};
};

namespace {

rosa_status fail(rosa_batch *b, rosa_status st, const std::string &msg) {
  if (b) b->last_error = msg;
  else g_create_error = msg;
  return st;
}

rosa_status device_fail(rosa_batch *b, hipError_t e, const char *what) {
  std::string msg = std::string(what) + ": " + hipGetErrorString(e);
  if (b) {
    b->poisoned = true;
    b->last_error = msg;
  } else {
    g_create_error = msg;
  }
  return ROSA_E_DEVICE;
}

rosa_status check_config(const rosa_model_config *c) {
  if (c->n_layers < 1 || c->d_model < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1 || c->head_dim < 1 ||
      c->d_mlp < 1 || c->action_dim < 1 || c->time_emb_dim < 2 || !(c->rms_eps >= 0.f))
    return ROSA_E_INVALID;
  if (c->dtype != ROSA_BF16 && c->dtype != ROSA_FP32) return ROSA_E_INVALID;
  if (c->attention_layout != ROSA_ATTN_JOINT && c->attention_layout != ROSA_ATTN_ALTERNATING) return ROSA_E_INVALID;
  if (c->n_q_heads % c->n_kv_heads != 0) return ROSA_E_UNSUPPORTED;
  if (c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 128 && c->head_dim != 256)
    return ROSA_E_UNSUPPORTED;
  if (c->d_model % 128 || c->d_mlp % 128 || (c->n_q_heads * c->head_dim) % 128) return ROSA_E_UNSUPPORTED;
  if (c->d_model > 4096 || c->action_dim > 64 || c->time_emb_dim % 2 || c->time_emb_dim > 8192)
    return ROSA_E_UNSUPPORTED;
  return ROSA_OK;
}

rosa_status check_capacity(const rosa_capacity *c) {
  if (c->max_requests < 1 || c->max_horizon < 1 || c->max_action_tokens < 1 || c->max_steps < 1 ||
      c->max_prefix_tokens < 0)
    return ROSA_E_INVALID;
  if (c->max_steps > kMaxSteps) return ROSA_E_UNSUPPORTED;
  return ROSA_OK;
}

Dims make_dims(const rosa_model_config *c) {
  Dims d{};
  d.L = c->n_layers; d.d = c->d_model; d.nq = c->n_q_heads; d.nkv = c->n_kv_heads; d.hd = c->head_dim;
  d.dff = c->d_mlp; d.A = c->action_dim; d.dt = c->time_emb_dim;
  d.qkv_dim = (d.nq + 2 * d.nkv) * d.hd;
  d.o_dim = d.nq * d.hd;
  d.mod_stride = d.L * 6 * d.d + 2 * d.d;
  d.eps = c->rms_eps;
  return d;
}

// Query blocks of R query rows: 32-row groups, at most `per` per block (4 per
// wave group of the bf16 kernel; the fp32 kernel takes any block).
int attn_query_blocks(int R, int per) { return ((R + 31) / 32 + per - 1) / per; }
int attn_groups_per_block(const rosa_model_config *cfg) { return 4 * attn_groups_per_wave(cfg->head_dim); }

// Attention set of a layer: 0 for joint layers and the alternating layout's
// cross-attention (even) layers, 1 for its self-attention (odd) layers.
int attn_set_of(const rosa_model_config *cfg, int layer) {
  return cfg->attention_layout == ROSA_ATTN_ALTERNATING && (layer & 1) ? 1 : 0;
}

// Validation of a request set (all-or-nothing) and the batch plan.
rosa_status build_plan(const rosa_model_config *cfg, const rosa_capacity *cap, const rosa_request *reqs,
                       int n, bool sort_by_steps, bool allow_split, int lanes_wanted, Plan &p, std::string &err,
                       int max_steps_call = INT32_MAX, int max_slots = -1) {
  if (n < 0) { err = "n_reqs < 0"; return ROSA_E_INVALID; }
  if (n > 0 && !reqs) { err = "reqs is NULL"; return ROSA_E_INVALID; }
  if (n > cap->max_requests) { err = "more requests than max_requests"; return ROSA_E_CAPACITY; }
  int64_t sumH = 0, sumP = 0;
  for (int i = 0; i < n; ++i) {
    const rosa_request &r = reqs[i];
    char buf[160];
    if (r.prefix_len < 0 || r.horizon < 1 || r.num_steps < 1) {
      snprintf(buf, sizeof buf, "request %d: P=%d H=%d K=%d out of range", i, r.prefix_len, r.horizon, r.num_steps);
      err = buf; return ROSA_E_INVALID;
    }
    if (r.horizon > cap->max_horizon || r.num_steps > cap->max_steps) {
      snprintf(buf, sizeof buf, "request %d: H=%d or K=%d above max_horizon=%d / max_steps=%d", i, r.horizon,
               r.num_steps, cap->max_horizon, cap->max_steps);
      err = buf; return ROSA_E_INVALID;
    }
    if (r.start_step < 0 || r.start_step >= r.num_steps) {
      snprintf(buf, sizeof buf, "request %d: start_step=%d outside [0, K=%d)", i, r.start_step, r.num_steps);
      err = buf; return ROSA_E_INVALID;
    }
    if ((r.start_step == 0 && !r.noise) || !r.actions || (r.prefix_len > 0 && (!r.prefix_k || !r.prefix_v))) {
      snprintf(buf, sizeof buf, "request %d: NULL pointer", i); err = buf; return ROSA_E_INVALID;
    }
    if (cfg->attention_layout == ROSA_ATTN_ALTERNATING && r.prefix_len < 1) {
      snprintf(buf, sizeof buf, "request %d: the alternating layout needs a prefix (P >= 1)", i);
      err = buf; return ROSA_E_INVALID;
    }
    sumH += r.horizon;
    sumP += r.prefix_len;
  }
  if (sumH > cap->max_action_tokens) { err = "sum of horizons above max_action_tokens"; return ROSA_E_CAPACITY; }
  if (sumP > cap->max_prefix_tokens) { err = "sum of prefix lengths above max_prefix_tokens"; return ROSA_E_CAPACITY; }

  if (max_steps_call < 1) { err = "max_steps < 1"; return ROSA_E_INVALID; }
  p = Plan();
  // Euler steps each request runs in this call (by caller index).
  std::vector<int> nsteps(n);
  for (int i = 0; i < n; ++i) nsteps[i] = std::min(reqs[i].num_steps - reqs[i].start_step, max_steps_call);
  // Lanes: requests dealt longest-first to the lane with the least estimated
  // work (token-steps weighted by the attention's key count), then each lane
  // sorted by step count, descending (stable).
  const int n_lanes = std::max(1, std::min(lanes_wanted, n));
  std::vector<int> lane_of(n, 0);
  if (n_lanes > 1) {
    std::vector<int> byw(n);
    for (int i = 0; i < n; ++i) byw[i] = i;
    auto work = [&](int i) {
      const rosa_request &r = reqs[i];
      return (double)r.horizon * nsteps[i] * (1.0 + (double)(r.prefix_len + r.horizon) / 1800.0);
    };
    std::stable_sort(byw.begin(), byw.end(), [&](int a, int b2) { return work(a) > work(b2); });
    std::vector<double> load(n_lanes, 0.0);
    for (int i : byw) {
      int best = 0;
      for (int l = 1; l < n_lanes; ++l)
        if (load[l] < load[best]) best = l;
      lane_of[i] = best;
      load[best] += work(i);
    }
  }
  p.order.clear();
  p.lanes.resize(n_lanes);
  for (int l = 0; l < n_lanes; ++l) {
    const size_t lo = p.order.size();
    for (int i = 0; i < n; ++i)
      if (lane_of[i] == l) p.order.push_back(i);
    if (sort_by_steps)
      std::stable_sort(p.order.begin() + lo, p.order.end(),
                       [&](int a, int b2) { return nsteps[a] > nsteps[b2]; });
    p.lanes[l].req_lo = (int)lo;
    p.lanes[l].req_hi = (int)p.order.size();
  }
  p.tok_off.resize(n);
  int M = 0;
  p.steps.resize(n);
  for (int i = 0; i < n; ++i) {
    p.tok_off[i] = M;
    M += reqs[p.order[i]].horizon;
    p.steps[i] = nsteps[p.order[i]];
    p.Kmax = std::max(p.Kmax, p.steps[i]);
  }
  p.M0 = M;
  p.m_k.assign(p.Kmax, 0);
  p.n_active.assign(p.Kmax, 0);
  for (int i = 0; i < n; ++i)
    for (int k = 0; k < p.steps[i]; ++k) { p.m_k[k] += reqs[p.order[i]].horizon; p.n_active[k] += 1; }
  for (Plan::Lane &ln : p.lanes) {
    ln.row_lo = ln.req_lo < n ? p.tok_off[ln.req_lo] : M;
    ln.row_hi = ln.req_hi < n ? p.tok_off[ln.req_hi] : M;
    ln.n_act.assign(p.Kmax, 0);
    ln.m.assign(p.Kmax, 0);
    for (int i = ln.req_lo; i < ln.req_hi; ++i)
      for (int k = 0; k < p.steps[i]; ++k) { ln.m[k] += reqs[p.order[i]].horizon; ln.n_act[k] += 1; }
  }

  // Distinct flow times tau = k / K (fp32 division) of every (call step j,
  // request) with k = start_step + j, and their indices.
  p.tau_idx.assign((size_t)p.Kmax * n, 0);
  for (int i = 0; i < n; ++i) {
    const int K = reqs[p.order[i]].num_steps, k0 = reqs[p.order[i]].start_step;
    for (int k = 0; k < p.steps[i]; ++k) {
      const float tau = (float)(k0 + k) / (float)K;
      int idx = -1;
      for (size_t j = 0; j < p.taus.size(); ++j)
        if (p.taus[j] == tau) { idx = (int)j; break; }
      if (idx < 0) {
        if ((int)p.taus.size() >= kMaxTau) { err = "more than 128 distinct flow times in one call"; return ROSA_E_CAPACITY; }
        idx = (int)p.taus.size();
        p.taus.push_back(tau);
      }
      p.tau_idx[(size_t)k * n + i] = idx;
    }
  }

  // Attention work items: per request and KV head, its query rows in blocks of
  // at most kAttnQB rows (32-row groups spread evenly over the blocks), over
  // the set's key range of the request's key sequence [prefix ; actions]:
  // set 0 all of it (joint) or the prefix (alternating), set 1 the actions.
  // Keys are split over several items only when the batch is too small to
  // fill the GPU.
  const int G = cfg->n_q_heads / cfg->n_kv_heads;
  const int gpb = attn_groups_per_block(cfg);
  const bool alternating = cfg->attention_layout == ROSA_ATTN_ALTERNATING;
  p.n_sets = alternating ? 2 : 1;
  int64_t total_qb = 0;
  for (int i = 0; i < n; ++i) total_qb += (int64_t)cfg->n_kv_heads * attn_query_blocks(reqs[i].horizon * G, gpb);
  // Partial-result slots available per attention set (every split item takes one).
  const int64_t slot_budget = (max_slots < 0 ? (int64_t)p.n_sets * kMaxSlots : (int64_t)max_slots) / p.n_sets;
  const int64_t want_all = total_qb > 0 ? (kSplitTarget + total_qb - 1) / total_qb : 1;
  const int64_t want_fit = total_qb > 0 ? slot_budget / total_qb : 0;
  const int want_split = (int)std::min(want_all, want_fit);
  const bool split = allow_split && total_qb > 0 && total_qb < kSplitTarget && want_split >= 2;
  for (int v = 0; v < p.n_sets; ++v) {
    Plan::AttnSet &S = p.sets[v];
    if (v == 1) { S.item_base = (int)p.sets[0].items.size(); S.group_base = (int)p.sets[0].groups.size(); }
    S.items_upto.resize(n);
    S.groups_upto.resize(n);
    for (int i = 0; i < n; ++i) {
      const rosa_request &r = reqs[p.order[i]];
      const int key_lo = v == 1 ? r.prefix_len : 0;
      const int key_hi = alternating && v == 0 ? r.prefix_len : r.prefix_len + r.horizon;
      const int nk = key_hi - key_lo;
      const int R = r.horizon * G, ngrp = (R + 31) / 32, nqb = attn_query_blocks(R, gpb);
      int nsplit = 1, chunk = nk;
      if (split) {
        const int want = want_split;
        const int most = std::max(1, (nk + kMinSplitKeys - 1) / kMinSplitKeys);
        nsplit = std::min(want, most);
        chunk = (nk + nsplit - 1) / nsplit;
        chunk = (chunk + 63) / 64 * 64;          // whole 64-key tiles per item
        nsplit = (nk + chunk - 1) / chunk;
      }
      for (int kvh = 0; kvh < cfg->n_kv_heads; ++kvh)
        for (int qb = 0; qb < nqb; ++qb) {
          const int q0 = 32 * (qb * ngrp / nqb);
          const int nq = std::min(R, 32 * ((qb + 1) * ngrp / nqb)) - q0;
          if (nsplit > 1) {
            AttnGroup gr{i, kvh, q0, nq, p.slots, nsplit, 0, 0};
            S.groups.push_back(gr);
          }
          for (int c = 0; c < nsplit; ++c) {
            AttnItem it{};
            it.pk = r.prefix_k; it.pv = r.prefix_v; it.P = r.prefix_len; it.tok_off = p.tok_off[i];
            it.req = i; it.kvh = kvh; it.q0 = q0; it.nq = nq;
            it.kbeg = key_lo + c * chunk;
            it.kend = std::min(key_hi, key_lo + (c + 1) * chunk);
            it.slot = nsplit > 1 ? p.slots++ : -1;
            S.items.push_back(it);
          }
        }
      S.items_upto[i] = (int)S.items.size();
      S.groups_upto[i] = (int)S.groups.size();
    }
  }
  if (p.slots > (max_slots < 0 ? p.n_sets * kMaxSlots : max_slots)) {
    err = "internal: attention partial slots exceeded";
    return ROSA_E_CAPACITY;
  }

  // Attention launch orders, one per set and distinct set of active requests
  // of a lane; entries index the whole device item array.
  for (Plan::Lane &ln : p.lanes)
    for (int v = 0; v < p.n_sets; ++v) {
      const Plan::AttnSet &S = p.sets[v];
      ln.list_at[v].assign(p.Kmax, -1);
      ln.list_blocks[v].assign(p.Kmax, 0);
      int prev_n = -1;
      for (int k = 0; k < p.Kmax; ++k) {
        const int na = ln.n_act[k];
        if (na == 0) continue;
        if (na == prev_n) {
          ln.list_at[v][k] = ln.list_at[v][k - 1];
          ln.list_blocks[v][k] = ln.list_blocks[v][k - 1];
          continue;
        }
        prev_n = na;
        std::vector<std::pair<int, int>> ranges;
        for (int i = ln.req_lo; i < ln.req_lo + na; ++i)
          ranges.push_back({i > 0 ? S.items_upto[i - 1] : 0, S.items_upto[i]});
        const size_t at = p.attn_lists.size();
        ln.list_at[v][k] = (int)at;
        ln.list_blocks[v][k] = attn_launch_order(S.items, ranges, p.attn_lists, p.attn_next);
        for (size_t e = at; e < p.attn_lists.size(); ++e)
          if (p.attn_lists[e] >= 0) p.attn_lists[e] += S.item_base;
      }
    }
  return ROSA_OK;
}

template <typename T>
T *dalloc(rosa_batch *b, size_t count, hipError_t &e) {
  void *ptr = nullptr;
  if (e != hipSuccess) return nullptr;
  e = hipMalloc(&ptr, std::max<size_t>(count * sizeof(T), 256));
  if (e == hipSuccess) b->allocations.push_back(ptr);
  return (T *)ptr;
}

// Upload a host fp32 tensor, converted to the activation dtype.
hipError_t upload_act(rosa_batch *b, void *dst, const float *src, size_t n) {
  if (!b->bf16) return hipMemcpy(dst, src, n * 4, hipMemcpyHostToDevice);
  std::vector<uint16_t> tmp(n);
  for (size_t i = 0; i < n; ++i) tmp[i] = f32_to_bf16_rne(src[i]);
  return hipMemcpy(dst, tmp.data(), n * 2, hipMemcpyHostToDevice);
}

// Upload L stacked [K][N] matrices as [L][N][K] (transposed), activation dtype.
hipError_t upload_transposed(rosa_batch *b, void *dst, const float *src, int L, int K, int N) {
  return upload_weights_transposed(dst, src, L, K, N, b->bf16);
}

// Profiling helpers.
hipEvent_t get_event(rosa_batch *b) {
  if (!b->free_events.empty()) { hipEvent_t e = b->free_events.back(); b->free_events.pop_back(); return e; }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

template <typename F>
hipError_t timed(rosa_batch *b, int cls, F &&launch) {
  if (!b->prof) return launch();
  hipEvent_t e0 = get_event(b), e1 = get_event(b);
  if (!e0 || !e1) return launch();
  hipEventRecord(e0, b->stream);
  const hipError_t err = launch();
  hipEventRecord(e1, b->stream);
  b->pending.push_back({cls, e0, e1});
  return err;
}

hipError_t harvest_profile(rosa_batch *b) {
  hipError_t e = hipStreamSynchronize(b->stream);
  if (e != hipSuccess) return e;
  for (auto &p : b->pending) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      b->prof_ms[p.cls] += ms;
      b->prof_launches[p.cls] += 1;
    }
    b->free_events.push_back(p.a);
    b->free_events.push_back(p.b);
  }
  b->pending.clear();
  return hipSuccess;
}

// Copy the plan through a pinned staging buffer into the device plan region.
hipError_t upload_plan(rosa_batch *b, const Plan &p, const rosa_request *reqs, int n) {
  const Plan::AttnSet &S0 = p.sets[0], &S1 = p.sets[1];
  const size_t n_items = S0.items.size() + S1.items.size(), n_groups = S0.groups.size() + S1.groups.size();
  if ((int64_t)n_items > b->max_items || (int64_t)n_groups > b->max_slots || p.attn_lists.size() > b->max_list_ints)
    return hipErrorInvalidValue;
  const int slot = b->plan_flip;
  b->plan_flip ^= 1;
  if (b->plan_pending[slot]) {
    hipError_t e = hipEventSynchronize(b->plan_copied[slot]);
    if (e != hipSuccess) return e;
  }
  uint8_t *hp = (uint8_t *)b->h_plan[slot];
  ReqDesc *rd = (ReqDesc *)(hp + b->off_reqs);
  for (int i = 0; i < n; ++i) {
    const rosa_request &r = reqs[p.order[i]];
    ReqDesc d{};
    d.pk = r.prefix_k; d.pv = r.prefix_v; d.noise = r.noise; d.actions = r.actions;
    d.P = r.prefix_len; d.H = r.horizon; d.K = r.num_steps; d.tok_off = p.tok_off[i]; d.orig = p.order[i];
    d.k0 = r.start_step; d.S = p.steps[i];
    rd[i] = d;
  }
  std::memcpy(hp + b->off_tau_idx, p.tau_idx.data(), p.tau_idx.size() * 4);
  std::memcpy(hp + b->off_taus, p.taus.data(), p.taus.size() * 4);
  std::memcpy(hp + b->off_items, S0.items.data(), S0.items.size() * sizeof(AttnItem));
  std::memcpy(hp + b->off_items + S0.items.size() * sizeof(AttnItem), S1.items.data(), S1.items.size() * sizeof(AttnItem));
  std::memcpy(hp + b->off_groups, S0.groups.data(), S0.groups.size() * sizeof(AttnGroup));
  std::memcpy(hp + b->off_groups + S0.groups.size() * sizeof(AttnGroup), S1.groups.data(),
              S1.groups.size() * sizeof(AttnGroup));
  {
    std::vector<AttnItem> all(S0.items);
    all.insert(all.end(), S1.items.begin(), S1.items.end());
    attn_order_items(all, p.attn_lists.data(), p.attn_next.data(), p.attn_lists.size(), (AttnItem *)(hp + b->off_lists));
  }
  const size_t used = b->off_lists + p.attn_lists.size() * sizeof(AttnItem);
  hipError_t e = hipMemcpyAsync(b->d_plan, hp, used, hipMemcpyHostToDevice, b->stream);
  if (e != hipSuccess) return e;
  e = hipEventRecord(b->plan_copied[slot], b->stream);
  b->plan_pending[slot] = true;
  return e;
}

// Modulation table for the plan's distinct flow times.
hipError_t run_time_conditioning(rosa_batch *b, const float *d_taus, int n_tau, float *out) {
  const Dims &D = b->dims;
  hipError_t e = timed(b, kcTime, [&] { return launch_time_embedding(d_taus, n_tau, D.dt, b->emb, b->stream); });
  if (e == hipSuccess)
    e = timed(b, kcTime, [&] { return launch_small_gemv(b->emb, n_tau, D.dt, b->w_t1, b->bf16, b->b_t1, D.d, 1, b->tc1, b->gemv_ws, b->stream); });
  if (e == hipSuccess)
    e = timed(b, kcTime, [&] { return launch_small_gemv(b->tc1, n_tau, D.d, b->w_t2, b->bf16, b->b_t2, D.d, 1, b->tc2, b->gemv_ws, b->stream); });
  if (e == hipSuccess)
    e = timed(b, kcTime, [&] { return launch_small_gemv(b->tc2, n_tau, D.d, b->w_modall, b->bf16, b->b_modall, D.mod_stride, 0, out, b->gemv_ws, b->stream); });
  return e;
}

// Attention of one layer for the requests active at step k of lane ln.
hipError_t run_attention(rosa_batch *b, const Plan &p, const Plan::Lane &ln, int k, int layer, const void *qkv,
                         void *o, hipStream_t st, int o_rows) {
  const Dims &D = b->dims;
  const ReqDesc *reqs = (const ReqDesc *)((uint8_t *)b->d_plan + b->off_reqs);
  const AttnItem *items = (const AttnItem *)((uint8_t *)b->d_plan + b->off_items);
  const AttnGroup *groups = (const AttnGroup *)((uint8_t *)b->d_plan + b->off_groups);
  const AttnItem *lists = (const AttnItem *)((uint8_t *)b->d_plan + b->off_lists);
  const int r0 = ln.req_lo, n_act = ln.n_act[k];
  if (n_act <= 0) return hipSuccess;
  const int v = attn_set_of(&b->cfg, layer);
  const Plan::AttnSet &S = p.sets[v];
  const int it_lo = S.item_base + (r0 > 0 ? S.items_upto[r0 - 1] : 0), it_hi = S.item_base + S.items_upto[r0 + n_act - 1];
  const int gr_lo = S.group_base + (r0 > 0 ? S.groups_upto[r0 - 1] : 0);
  const int gr_hi = S.group_base + S.groups_upto[r0 + n_act - 1];
  AttnArgs a{};
  a.items = items + it_lo; a.n_items = it_hi - it_lo;
  if (b->bf16) {   // launch order of this step's active set (indices into the whole item array)
    a.items = items;
    a.ordered = lists + ln.list_at[v][k];
    a.n_blocks = ln.list_blocks[v][k];
  }
  a.reqs = reqs; a.layer = layer;
  a.qkv = qkv; a.ldqkv = D.qkv_dim; a.o = o; a.ldo = D.o_dim; a.o_rows = o_rows;
  a.nq = D.nq; a.nkv = D.nkv; a.hd = D.hd;
  a.part_o = b->part_o; a.part_ml = b->part_ml;
  hipError_t e = timed(b, kcAttention, [&] { return launch_attention(a, b->bf16, st); });
  if (e == hipSuccess && gr_hi > gr_lo)
    e = timed(b, kcMerge, [&] {
      return launch_attn_merge(groups + gr_lo, gr_hi - gr_lo, reqs, b->part_o, b->part_ml, o, D.o_dim, D.nq, D.nkv,
                               D.hd, b->bf16, st, o_rows);
    });
  return e;
}

void free_all(rosa_batch *b) {
  for (void *ptr : b->allocations) hipFree(ptr);
  b->allocations.clear();
  for (int i = 0; i < 2; ++i) {
    if (b->h_plan[i]) hipHostFree(b->h_plan[i]);
    if (b->plan_copied[i]) hipEventDestroy(b->plan_copied[i]);
  }
  for (auto &p : b->pending) { hipEventDestroy(p.a); hipEventDestroy(p.b); }
  for (auto e : b->free_events) hipEventDestroy(e);
  for (int l = 1; l < kMaxLanes; ++l) {
    if (b->lane_stream[l]) hipStreamDestroy(b->lane_stream[l]);
    if (b->ev_join[l]) hipEventDestroy(b->ev_join[l]);
    b->lane_stream[l] = nullptr;
    b->ev_join[l] = nullptr;
  }
  if (b->ev_fork) hipEventDestroy(b->ev_fork);
  b->ev_fork = nullptr;
}

}  // namespace

// ====================================================================== allocation-free attention
// Scratch of rosa_attention_noalloc: the plan of a call (request descriptors,
// work items, merge groups, the block -> item table) and the partial results
// of key ranges split over several items.  One copy per GPU, held until the
// process ends; every call on a GPU reuses it (calls that overlap on one GPU
// race).  Nothing in it has to start at zero: each call uploads its plan and
// every partial slot is written by its item before the merge reads it.
namespace {
constexpr int kNaMaxRequests = 1024;
constexpr int kNaMaxItems = 4096;          // work items, and blocks of the launch order
constexpr int kNaMaxSlots = 64;            // partial-result slots (query blocks x key splits)
constexpr int kNaMaxHeadDim = 256;
constexpr size_t kNaOffReqs = 0;
constexpr size_t kNaOffItems = kNaOffReqs + (size_t)kNaMaxRequests * sizeof(ReqDesc);
constexpr size_t kNaOffGroups = kNaOffItems + (size_t)kNaMaxItems * sizeof(AttnItem);
constexpr size_t kNaOffLists = kNaOffGroups + (size_t)kNaMaxSlots * sizeof(AttnGroup);
constexpr size_t kNaOffMl = kNaOffLists + (size_t)kNaMaxItems * sizeof(AttnItem);
constexpr size_t kNaOffO = kNaOffMl + (size_t)kNaMaxSlots * kAttnQB * 2 * sizeof(float);
constexpr size_t kNaBytes = kNaOffO + (size_t)kNaMaxSlots * kAttnQB * kNaMaxHeadDim * sizeof(float);
static_assert(kNaOffItems % 256 == 0 && kNaOffGroups % 256 == 0 && kNaOffLists % 256 == 0 &&
              kNaOffMl % 256 == 0 && kNaOffO % 256 == 0, "scratch regions stay 256-byte aligned");
}  // namespace

static __device__ __align__(256) uint8_t scratch[kNaBytes];

namespace {
// Device address of `scratch` on the current device.  The array's name is a
// host-side stand-in in host code; the address comes from the runtime, once
// per device (with that device current), and is cached.
hipError_t noalloc_scratch(int dev, uint8_t **out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static uint8_t *addr[kMaxDevices] = {};
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    addr[dev] = static_cast<uint8_t *>(ptr);
  }
  *out = addr[dev];
  return hipSuccess;
}
}  // namespace

// ====================================================================== C ABI

extern "C" {

const char *rosa_status_string(rosa_status s) {
  // A C caller may pass any int; read it as one (loading an out-of-range
  // value through the enum type is undefined in C++).
  int v;
  std::memcpy(&v, &s, sizeof v);
  switch (v) {
    case ROSA_OK: return "ok";
    case ROSA_E_INVALID: return "invalid argument";
    case ROSA_E_CAPACITY: return "capacity exceeded";
    case ROSA_E_NOMEM: return "out of memory";
    case ROSA_E_DEVICE: return "device error";
    case ROSA_E_UNSUPPORTED: return "unsupported shape";
  }
  return "unknown status";
}

const char *rosa_last_error(const rosa_batch *b) {
  return b ? b->last_error.c_str() : g_create_error.c_str();
}

rosa_status rosa_batch_create(const rosa_model_config *cfg, const rosa_weights *w, const rosa_capacity *cap,
                              void *hip_stream, rosa_batch **out) {
  try {
    g_create_error.clear();
    if (!out) return fail(nullptr, ROSA_E_INVALID, "out is NULL");
    *out = nullptr;
    if (!cfg || !w || !cap) return fail(nullptr, ROSA_E_INVALID, "NULL config, weights or capacity");
    rosa_status st = check_config(cfg);
    if (st != ROSA_OK) return fail(nullptr, st, "model configuration not supported");
    st = check_capacity(cap);
    if (st != ROSA_OK) return fail(nullptr, st, "bad capacity");
    // a request's query rows (horizon x query heads per KV head) are int32 in the plan and kernels
    if ((int64_t)cap->max_horizon * (cfg->n_q_heads / cfg->n_kv_heads) > (int64_t(1) << 30))
      return fail(nullptr, ROSA_E_UNSUPPORTED, "max_horizon x query heads per KV head above 2^30");
    const float *need[] = {w->w_in, w->b_in, w->w_t1, w->b_t1, w->w_t2, w->b_t2, w->w_mod, w->b_mod, w->w_qkv,
                           w->w_o, w->w_up, w->w_down, w->w_fmod, w->b_fmod, w->w_out, w->b_out};
    for (const float *p : need)
      if (!p) return fail(nullptr, ROSA_E_INVALID, "NULL weight pointer");

    rosa_batch *b = new rosa_batch();
    b->cfg = *cfg;
    b->cap = *cap;
    b->dims = make_dims(cfg);
    b->bf16 = cfg->dtype == ROSA_BF16;
    b->esz = b->bf16 ? 2 : 4;
    b->stream = (hipStream_t)hip_stream;
    const Dims &D = b->dims;
    hipError_t e = hipGetDevice(&b->device);
    if (e != hipSuccess) { rosa_status s2 = device_fail(nullptr, e, "hipGetDevice"); delete b; return s2; }

    const size_t L = D.L, d = D.d, maxM = cap->max_action_tokens;
    // weights
    b->w_in = dalloc<float>(b, (size_t)D.A * d, e);
    b->b_in = dalloc<float>(b, d, e);
    b->w_t1 = dalloc<uint8_t>(b, (size_t)D.dt * d * b->esz, e);
    b->b_t1 = dalloc<float>(b, d, e);
    b->w_t2 = dalloc<uint8_t>(b, d * d * b->esz, e);
    b->b_t2 = dalloc<float>(b, d, e);
    b->w_modall = dalloc<uint8_t>(b, d * D.mod_stride * b->esz, e);
    b->b_modall = dalloc<float>(b, D.mod_stride, e);
    b->wt_qkv = dalloc<uint8_t>(b, L * D.qkv_dim * d * b->esz, e);
    b->wt_o = dalloc<uint8_t>(b, L * d * D.o_dim * b->esz, e);
    b->wt_up = dalloc<uint8_t>(b, L * D.dff * d * b->esz, e);
    b->wt_down = dalloc<uint8_t>(b, L * d * D.dff * b->esz, e);
    b->w_out = dalloc<float>(b, d * D.A, e);
    b->b_out = dalloc<float>(b, D.A, e);
    if (b->bf16) b->wt_out = dalloc<uint8_t>(b, (size_t)d * D.A * 2, e);
    // workspaces
    b->kb_rows = b->bf16 ? (int)maxM : 0;
    b->x = dalloc<float>(b, maxM * D.A, e);
    b->h = dalloc<float>(b, maxM * d, e);
    b->u = dalloc<uint8_t>(b, maxM * d * b->esz, e);
    b->qkv = dalloc<uint8_t>(b, maxM * D.qkv_dim * b->esz, e);
    b->o = dalloc<uint8_t>(b, maxM * D.o_dim * b->esz, e);
    b->g = dalloc<uint8_t>(b, maxM * D.dff * b->esz, e);
    b->row_req = dalloc<int32_t>(b, maxM, e);
    b->rowmod = dalloc<int32_t>(b, maxM * cap->max_steps, e);
    b->ident = dalloc<int32_t>(b, maxM, e);
    b->modtab = dalloc<float>(b, (size_t)kMaxTau * D.mod_stride, e);
    b->emb = dalloc<float>(b, (size_t)kMaxTau * D.dt, e);
    b->tc1 = dalloc<float>(b, (size_t)kMaxTau * d, e);
    b->tc2 = dalloc<float>(b, (size_t)kMaxTau * d, e);
    b->gemv_ws = dalloc<float>(b, small_gemv_workspace_floats(std::max(D.mod_stride, D.d)), e);
    const int n_sets = cfg->attention_layout == ROSA_ATTN_ALTERNATING ? 2 : 1;
    b->max_slots = n_sets * kMaxSlots;
    b->gemm_part_floats = b->bf16 ? std::min<size_t>((size_t)kSplitMax * maxM * std::max(D.qkv_dim, std::max(D.dff, D.d)),
                                                     (size_t)16 << 20)
                                  : 0;
    if (b->gemm_part_floats) b->gemm_part = dalloc<float>(b, b->gemm_part_floats, e);
    if (b->bf16) {
      b->dn_ss = dalloc<float>(b, maxM * (D.d / 32), e);
      b->dn_shift = dalloc<float>(b, (size_t)D.L * kMaxTau * (D.qkv_dim + D.dff), e);
    }
    b->part_o = dalloc<float>(b, (size_t)b->max_slots * kAttnQB * D.hd, e);
    b->part_ml = dalloc<float>(b, (size_t)b->max_slots * kAttnQB * 2, e);

    // plan region
    const int G = D.nq / D.nkv;
    const int64_t qb_bound = (int64_t)D.nkv * (((int64_t)maxM * G + 127) / 128 + 2 * (int64_t)cap->max_requests);
    b->max_items = (int)(n_sets * (kMaxSlots + qb_bound));
    auto align = [](size_t v) { return (v + 255) / 256 * 256; };
    b->off_reqs = 0;
    b->off_tau_idx = align(b->off_reqs + (size_t)cap->max_requests * sizeof(ReqDesc));
    b->off_taus = align(b->off_tau_idx + (size_t)cap->max_requests * cap->max_steps * 4);
    b->off_items = align(b->off_taus + kMaxTau * 4);
    b->off_groups = align(b->off_items + (size_t)b->max_items * sizeof(AttnItem));
    b->off_lists = align(b->off_groups + (size_t)b->max_slots * sizeof(AttnGroup));
    // one launch order per step and lane at most: its items plus at most as
    // many idle first entries (n_blocks <= items + 7)
    b->max_list_ints = (size_t)cap->max_steps * (2 * (size_t)b->max_items + 8 * kMaxLanes * n_sets);
    b->plan_bytes = align(b->off_lists + b->max_list_ints * sizeof(AttnItem));
    b->d_plan = dalloc<uint8_t>(b, b->plan_bytes, e);
    if (e != hipSuccess) {
      rosa_status s2 = e == hipErrorOutOfMemory ? fail(nullptr, ROSA_E_NOMEM, "device allocation failed")
                                                 : device_fail(nullptr, e, "hipMalloc");
      free_all(b); delete b; return s2;
    }
    for (int i = 0; i < 2 && e == hipSuccess; ++i) {
      e = hipHostMalloc(&b->h_plan[i], b->plan_bytes, hipHostMallocDefault);
      if (e == hipSuccess) e = hipEventCreateWithFlags(&b->plan_copied[i], hipEventDisableTiming);
    }
    b->lanes = b->bf16 ? 2 : 1;
    b->lane_stream[0] = b->stream;
    if (e == hipSuccess) e = hipEventCreateWithFlags(&b->ev_fork, hipEventDisableTiming);
    for (int l = 1; l < kMaxLanes && e == hipSuccess; ++l) {
      e = hipStreamCreateWithFlags(&b->lane_stream[l], hipStreamNonBlocking);
      if (e == hipSuccess) e = hipEventCreateWithFlags(&b->ev_join[l], hipEventDisableTiming);
    }
    if (e != hipSuccess) { rosa_status s2 = fail(nullptr, ROSA_E_NOMEM, "pinned host allocation failed"); free_all(b); delete b; return s2; }

    // upload weights
    std::vector<float> modall(d * D.mod_stride), bmodall(D.mod_stride);
    for (size_t l = 0; l < L; ++l)
      for (size_t i = 0; i < d; ++i)
        std::memcpy(&modall[i * D.mod_stride + l * 6 * d], w->w_mod + (l * d + i) * 6 * d, 6 * d * 4);
    for (size_t i = 0; i < d; ++i)
      std::memcpy(&modall[i * D.mod_stride + L * 6 * d], w->w_fmod + i * 2 * d, 2 * d * 4);
    std::memcpy(bmodall.data(), w->b_mod, L * 6 * d * 4);
    std::memcpy(bmodall.data() + L * 6 * d, w->b_fmod, 2 * d * 4);
    if (e == hipSuccess) e = hipMemcpy(b->w_in, w->w_in, (size_t)D.A * d * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(b->b_in, w->b_in, d * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = upload_act(b, b->w_t1, w->w_t1, (size_t)D.dt * d);
    if (e == hipSuccess) e = hipMemcpy(b->b_t1, w->b_t1, d * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = upload_act(b, b->w_t2, w->w_t2, d * d);
    if (e == hipSuccess) e = hipMemcpy(b->b_t2, w->b_t2, d * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = upload_act(b, b->w_modall, modall.data(), modall.size());
    if (e == hipSuccess) e = hipMemcpy(b->b_modall, bmodall.data(), bmodall.size() * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = upload_gemm_weights(b->wt_qkv, w->w_qkv, D.L, D.d, D.qkv_dim, b->bf16);
    if (e == hipSuccess) e = upload_gemm_weights(b->wt_o, w->w_o, D.L, D.o_dim, D.d, b->bf16);
    if (e == hipSuccess) e = upload_gemm_weights(b->wt_up, w->w_up, D.L, D.d, D.dff, b->bf16);
    if (e == hipSuccess) e = upload_gemm_weights(b->wt_down, w->w_down, D.L, D.dff, D.d, b->bf16);
    if (e == hipSuccess) e = hipMemcpy(b->w_out, w->w_out, d * D.A * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(b->b_out, w->b_out, D.A * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess && b->bf16) e = upload_transposed(b, b->wt_out, w->w_out, 1, D.d, D.A);
    if (e == hipSuccess) {
      std::vector<int32_t> id(maxM);
      for (size_t i = 0; i < maxM; ++i) id[i] = (int32_t)i;
      e = hipMemcpy(b->ident, id.data(), maxM * 4, hipMemcpyHostToDevice);
    }
    if (e != hipSuccess) { rosa_status s2 = device_fail(nullptr, e, "weight upload"); free_all(b); delete b; return s2; }
    *out = b;
    return ROSA_OK;
  } catch (const std::bad_alloc &) {
    return fail(nullptr, ROSA_E_NOMEM, "host allocation failed");
  } catch (...) {
    return fail(nullptr, ROSA_E_DEVICE, "unexpected exception");
  }
}

rosa_status rosa_generate_actions(rosa_batch *b, const rosa_request *reqs, int32_t n) {
  return rosa_generate_steps(b, reqs, n, INT32_MAX);
}

rosa_status rosa_generate_steps(rosa_batch *b, const rosa_request *reqs, int32_t n, int32_t max_steps) {
  if (!b) return ROSA_E_INVALID;
  try {
    b->last_error.clear();
    if (b->poisoned) return fail(b, ROSA_E_DEVICE, "handle is poisoned by an earlier device error");
    Plan p;
    std::string err;
    // Lanes only without per-kernel profiling (its events live on one stream)
    // and with enough requests for each lane.
    const int lanes = b->prof ? 1 : std::max(1, std::min(b->lanes, n / kMinLaneRequests));
    rosa_status st = build_plan(&b->cfg, &b->cap, reqs, n, true, b->bf16, lanes, p, err, max_steps);
    if (st != ROSA_OK) return fail(b, st, err);
    if (n == 0) return ROSA_OK;
    hipError_t e = hipSetDevice(b->device);
    if (e == hipSuccess) e = upload_plan(b, p, reqs, n);
    if (e != hipSuccess) return device_fail(b, e, "plan upload");
    const Dims &D = b->dims;
    uint8_t *dp = (uint8_t *)b->d_plan;
    const ReqDesc *d_reqs = (const ReqDesc *)(dp + b->off_reqs);
    const int32_t *d_tau_idx = (const int32_t *)(dp + b->off_tau_idx);
    const float *d_taus = (const float *)(dp + b->off_taus);

    e = run_time_conditioning(b, d_taus, (int)p.taus.size(), b->modtab);
    if (e == hipSuccess)
      e = timed(b, kcSetup, [&] {
        return launch_setup_rows(d_reqs, n, d_tau_idx, p.Kmax, D.A, b->row_req, b->rowmod, p.M0, b->x, b->stream);
      });
    const int nl = (int)p.lanes.size();
    // Deferred norms: every unsplit output projection and MLP-down leaves t
    // and the row sums of squares for the next product, which completes the
    // norm; the shift halves are computed once per call, when some launch of
    // the call takes that path.
    const int n_tau = (int)p.taus.size();
    bool defer_on = false;
    if (b->bf16 && b->dn_ss && b->kb_rows > 0 && D.d % 256 == 0 && D.d <= 1024) {
      for (const Plan::Lane &ln : p.lanes)
        for (int k = 0; k < p.Kmax && !defer_on; ++k) {
          if (ln.m[k] == 0 || ln.m[k] > kDeferMaxRows) continue;
          GemmArgs t{};
          if (nl == 1) { t.part = b->gemm_part; t.part_floats = b->gemm_part_floats; }
          t.M = ln.m[k]; t.N = D.d; t.ldo = D.d; t.epi = kEpiGatedResidual;
          const NormArgs nm{b->modtab, D.mod_stride, 0, 0, D.eps, b->u, b->kb_rows};
          for (int K2 : {D.o_dim, D.dff}) {
            t.K = K2;
            if (gemm_defers(t, b->gemm_cfg, &nm)) defer_on = true;
          }
        }
    }
    const int n_dn = D.qkv_dim + D.dff;
    if (e == hipSuccess && defer_on)
      e = timed(b, kcTime, [&] {
        return launch_shift_proj(b->modtab, D.mod_stride, n_tau, D.L, 6 * D.d, 0, 3 * D.d, D.d, b->wt_qkv, D.qkv_dim,
                                 b->wt_up, D.dff, b->dn_shift, b->stream);
      });
    // Fork: every other lane's stream waits for the plan, the modulation table
    // and the row setup.
    if (e == hipSuccess && nl > 1) {
      e = hipEventRecord(b->ev_fork, b->stream);
      for (int li = 1; li < nl && e == hipSuccess; ++li) e = hipStreamWaitEvent(b->lane_stream[li], b->ev_fork, 0);
    }
    const size_t d6 = (size_t)6 * D.d;
    const size_t es = b->esz;
    for (int k = 0; k < p.Kmax && e == hipSuccess; ++k) {
      for (int li = 0; li < nl && e == hipSuccess; ++li) {
        const Plan::Lane &ln = p.lanes[li];
        const int M = ln.m[k];
        const int n_act = ln.n_act[k];
        if (M == 0) continue;
        const hipStream_t st = b->lane_stream[li];
        const size_t r0 = (size_t)ln.row_lo;
        // This lane's rows of every per-row buffer.
        // (kb32 operands: a lane's rows start r0 rows into every 32-wide plane.)
        const int R = b->kb_rows;
        float *x = b->x + r0 * D.A, *h = b->h + r0 * D.d;
        uint8_t *u = (uint8_t *)b->u + r0 * (R ? 32 : D.d) * es, *qkv = (uint8_t *)b->qkv + r0 * D.qkv_dim * es;
        uint8_t *o = (uint8_t *)b->o + r0 * (R ? 32 : D.o_dim) * es, *g = (uint8_t *)b->g + r0 * (R ? 32 : D.dff) * es;
        const int32_t *rowmod = b->rowmod + (size_t)k * p.M0 + r0;
        const int32_t *row_req = b->row_req + r0;
        e = timed(b, kcInProj, [&] { return launch_in_proj(x, M, D.A, b->w_in, b->b_in, D.d, h, st); });
        const int fshift = D.L * (int)d6, fscale = D.L * (int)d6 + D.d;
        float *dss = defer_on && M <= kDeferMaxRows ? b->dn_ss + r0 * (D.d / 32) : nullptr;
        // The deferred norm's producer outputs (t into u) and its completion
        // in the product that reads u, from this layer's shift table.
        auto defer_out = [&](GemmArgs &gx, int scale_off) {
          if (!dss) return;
          gx.dt = u; gx.dt_rows = R; gx.dss = dss; gx.dscale = b->modtab + scale_off;
        };
        auto defer_in = [&](GemmArgs &gx, int l2, int col0) {
          gx.css = dss; gx.cparts = D.d / 32; gx.cd = D.d; gx.ceps = D.eps; gx.rowmod = rowmod;
          gx.cshift = b->dn_shift + (size_t)l2 * n_tau * n_dn + col0; gx.cshift_stride = n_dn;
        };
        // u_ready: the norm that reads the rows just updated was fused into
        // the split product that updated them (small batches only); t_ready:
        // u holds that norm's deferred form (t, and the row sums in dss).
        bool u_ready = false, t_ready = false;
        for (int l = 0; l < D.L && e == hipSuccess; ++l) {
          const int base = (int)(l * d6);
          if (!u_ready && !t_ready)
            e = timed(b, kcModNorm, [&] {
              return launch_modnorm(h, M, D.d, D.eps, b->modtab, D.mod_stride, base, base + D.d, rowmod, u, b->bf16,
                                    st, R);
            });
          if (e != hipSuccess) break;
          GemmArgs gq{};
          if (nl == 1) { gq.part = b->gemm_part; gq.part_floats = b->gemm_part_floats; }
          gq.a = u; gq.lda = D.d; gq.a_rows = R; gq.wt = (uint8_t *)b->wt_qkv + (size_t)l * D.qkv_dim * D.d * es;
          gq.M = M; gq.N = D.qkv_dim; gq.K = D.d; gq.epi = kEpiStore; gq.out = qkv; gq.ldo = D.qkv_dim;
          if (t_ready) defer_in(gq, l, 0);
          u_ready = t_ready = false;
          e = timed(b, kcGemmQKV, [&] { return launch_gemm(gq, b->bf16, st, b->gemm_cfg); });
          if (e != hipSuccess) break;
          e = run_attention(b, p, ln, k, l, b->qkv, b->o, st, b->kb_rows);
          if (e != hipSuccess) break;
          GemmArgs go{};
          if (nl == 1) { go.part = b->gemm_part; go.part_floats = b->gemm_part_floats; }
          go.a = o; go.lda = D.o_dim; go.a_rows = R; go.wt = (uint8_t *)b->wt_o + (size_t)l * D.d * D.o_dim * es;
          go.M = M; go.N = D.d; go.K = D.o_dim; go.epi = kEpiGatedResidual; go.out = h; go.ldo = D.d;
          go.gate = b->modtab + base + 2 * D.d; go.gate_stride = D.mod_stride; go.rowmod = rowmod;
          const NormArgs mlp_norm{b->modtab, D.mod_stride, base + 3 * D.d, base + 4 * D.d, D.eps, u, R};
          defer_out(go, base + 4 * D.d);
          e = timed(b, kcGemmO, [&] { return launch_gemm(go, b->bf16, st, b->gemm_cfg, &mlp_norm, &u_ready, &t_ready); });
          if (e != hipSuccess) break;
          if (!u_ready && !t_ready)
            e = timed(b, kcModNorm, [&] {
              return launch_modnorm(h, M, D.d, D.eps, b->modtab, D.mod_stride, base + 3 * D.d, base + 4 * D.d, rowmod,
                                    u, b->bf16, st, R);
            });
          if (e != hipSuccess) break;
          GemmArgs gu{};
          if (nl == 1) { gu.part = b->gemm_part; gu.part_floats = b->gemm_part_floats; }
          gu.a = u; gu.lda = D.d; gu.a_rows = R; gu.out_rows = R; gu.wt = (uint8_t *)b->wt_up + (size_t)l * D.dff * D.d * es;
          gu.M = M; gu.N = D.dff; gu.K = D.d; gu.epi = kEpiGelu; gu.out = g; gu.ldo = D.dff;
          if (t_ready) defer_in(gu, l, D.qkv_dim);
          u_ready = t_ready = false;
          e = timed(b, kcGemmUp, [&] { return launch_gemm(gu, b->bf16, st, b->gemm_cfg); });
          if (e != hipSuccess) break;
          GemmArgs gd{};
          if (nl == 1) { gd.part = b->gemm_part; gd.part_floats = b->gemm_part_floats; }
          gd.a = g; gd.lda = D.dff; gd.a_rows = R; gd.wt = (uint8_t *)b->wt_down + (size_t)l * D.d * D.dff * es;
          gd.M = M; gd.N = D.d; gd.K = D.dff; gd.epi = kEpiGatedResidual; gd.out = h; gd.ldo = D.d;
          gd.gate = b->modtab + base + 5 * D.d; gd.gate_stride = D.mod_stride; gd.rowmod = rowmod;
          // The next norm: the next layer's attention norm, or the final norm.
          const bool last = l + 1 == D.L;
          const NormArgs next_norm{b->modtab, D.mod_stride, last ? fshift : base + (int)d6,
                                   last ? fscale : base + (int)d6 + D.d, D.eps, u, R};
          if (!last) defer_out(gd, base + (int)d6 + D.d);
          e = timed(b, kcGemmDown, [&] {
            return launch_gemm(gd, b->bf16, st, b->gemm_cfg, &next_norm, &u_ready, &t_ready);
          });
        }
        // Final norm with the final modulation, output projection and Euler step.
        if (e == hipSuccess && b->bf16) {
          if (!u_ready)
            e = timed(b, kcFinal, [&] {
              return launch_modnorm(h, M, D.d, D.eps, b->modtab, D.mod_stride, fshift, fscale, rowmod, u, true, st, R);
            });
          if (e == hipSuccess)
            e = timed(b, kcFinal, [&] {
              return launch_out_proj_euler((const __bf16 *)u, M, D.d, (const __bf16 *)b->wt_out, b->b_out, D.A, row_req,
                                           d_reqs, k, x, (int)r0, st, R);
            });
        } else if (e == hipSuccess) {
          e = timed(b, kcFinal, [&] {
            return launch_final_euler(h, M, D.d, D.eps, b->modtab, D.mod_stride, fshift, fscale, rowmod, b->w_out,
                                      b->b_out, D.A, row_req, d_reqs, k, x, (int)r0, st);
          });
        }
      }
    }
    // Join: the caller's stream waits for every lane.  After a failed launch
    // the lanes are still joined (and then drained), so that no lane can be
    // reading the caller's buffers or the handle's workspaces once the call
    // has returned its error.
    const hipError_t launch_err = e;
    hipError_t join_err = hipSuccess;
    for (int li = 1; li < nl; ++li) {
      hipError_t j = hipEventRecord(b->ev_join[li], b->lane_stream[li]);
      if (j == hipSuccess) j = hipStreamWaitEvent(b->stream, b->ev_join[li], 0);
      if (j != hipSuccess && join_err == hipSuccess) join_err = j;
    }
    if (launch_err != hipSuccess || join_err != hipSuccess) {
      for (int li = 0; li < nl; ++li) (void)hipStreamSynchronize(b->lane_stream[li]);
      return device_fail(b, launch_err != hipSuccess ? launch_err : join_err, "kernel launch");
    }
    return ROSA_OK;
  } catch (const std::bad_alloc &) {
    return fail(b, ROSA_E_NOMEM, "host allocation failed");
  } catch (...) {
    return fail(b, ROSA_E_DEVICE, "unexpected exception");
  }
}

void rosa_destroy(rosa_batch *b) {
  if (!b) return;
  try {
    hipSetDevice(b->device);
    hipStreamSynchronize(b->stream);
    for (int l = 1; l < kMaxLanes; ++l)
      if (b->lane_stream[l]) hipStreamSynchronize(b->lane_stream[l]);
    free_all(b);
  } catch (...) {
  }
  delete b;
}

// ---------------------------------------------------------------------- debug ABI

rosa_status rosa_debug_plan(const rosa_model_config *cfg, const rosa_capacity *cap, const rosa_request *reqs,
                            int32_t n, int32_t *order, int32_t *tok_off, int32_t *m_k, int32_t *counts) {
  try {
    if (!cfg || !cap) return ROSA_E_INVALID;
    rosa_status st = check_config(cfg);
    if (st != ROSA_OK) return st;
    st = check_capacity(cap);
    if (st != ROSA_OK) return st;
    Plan p;
    std::string err;
    st = build_plan(cfg, cap, reqs, n, true, cfg->dtype == ROSA_BF16, 1, p, err);
    if (st != ROSA_OK) return st;
    for (int i = 0; i < n; ++i) {
      if (order) order[i] = p.order[i];
      if (tok_off) tok_off[p.order[i]] = p.tok_off[i];
    }
    if (m_k)
      for (int k = 0; k < cap->max_steps; ++k) m_k[k] = k < p.Kmax ? p.m_k[k] : 0;
    if (counts) {
      counts[0] = (int32_t)p.taus.size();
      counts[1] = (int32_t)(p.sets[0].items.size() + p.sets[1].items.size());
      counts[2] = 0;
      for (int i = 0; i < n; ++i) {
        const int G = cfg->n_q_heads / cfg->n_kv_heads;
        counts[2] += cfg->n_kv_heads * attn_query_blocks(reqs[i].horizon * G, attn_groups_per_block(cfg));
      }
      counts[3] = (int32_t)(p.sets[0].groups.size() + p.sets[1].groups.size());
    }
    return ROSA_OK;
  } catch (...) {
    return ROSA_E_NOMEM;
  }
}

rosa_status rosa_debug_attn_lists(const rosa_model_config *cfg, const rosa_capacity *cap, const rosa_request *reqs,
                                  int32_t n, int32_t max_entries, int32_t *n_blocks, int32_t *n_entries,
                                  int32_t *item_of, int32_t *next, int32_t *item_cost) {
  try {
    if (!cfg || !cap || !n_blocks || !n_entries || max_entries < 0) return ROSA_E_INVALID;
    if (cfg->dtype != ROSA_BF16) return ROSA_E_UNSUPPORTED;
    rosa_status st = check_config(cfg);
    if (st != ROSA_OK) return st;
    st = check_capacity(cap);
    if (st != ROSA_OK) return st;
    Plan p;
    std::string err;
    st = build_plan(cfg, cap, reqs, n, true, true, 1, p, err);
    if (st != ROSA_OK) return st;
    *n_blocks = 0;
    *n_entries = 0;
    if (p.lanes.empty() || p.Kmax == 0 || p.lanes[0].list_at[0].empty() || p.lanes[0].list_at[0][0] < 0) return ROSA_OK;
    const Plan::Lane &ln = p.lanes[0];
    const size_t lo = (size_t)ln.list_at[0][0];
    size_t hi = p.attn_lists.size();
    for (int k = 1; k < p.Kmax; ++k)
      if (ln.list_at[0][k] > (int)lo) { hi = (size_t)ln.list_at[0][k]; break; }
    if (p.n_sets > 1 && !ln.list_at[1].empty() && ln.list_at[1][0] > (int)lo) hi = std::min(hi, (size_t)ln.list_at[1][0]);
    *n_blocks = ln.list_blocks[0][0];
    *n_entries = (int32_t)(hi - lo);
    if ((int64_t)(hi - lo) > max_entries) return ROSA_E_CAPACITY;
    for (size_t e = lo; e < hi; ++e) {
      if (item_of) item_of[e - lo] = p.attn_lists[e];
      if (next) next[e - lo] = p.attn_next[e];
    }
    if (item_cost)
      for (size_t i = 0; i < p.sets[0].items.size(); ++i) {
        const AttnItem &it = p.sets[0].items[i];
        item_cost[i] = (it.kend - it.kbeg + 31) / 32;
      }
    return ROSA_OK;
  } catch (...) {
    return ROSA_E_NOMEM;
  }
}

rosa_status rosa_debug_plan_lanes(const rosa_model_config *cfg, const rosa_capacity *cap, const rosa_request *reqs,
                                  int32_t n, int32_t lanes, int32_t *lane_of) {
  try {
    if (!cfg || !cap || !lane_of || lanes < 1 || lanes > kMaxLanes) return ROSA_E_INVALID;
    rosa_status st = check_config(cfg);
    if (st != ROSA_OK) return st;
    st = check_capacity(cap);
    if (st != ROSA_OK) return st;
    const int nl = cfg->dtype == ROSA_BF16 ? std::max(1, std::min<int>(lanes, n / kMinLaneRequests)) : 1;
    Plan p;
    std::string err;
    st = build_plan(cfg, cap, reqs, n, true, cfg->dtype == ROSA_BF16, nl, p, err);
    if (st != ROSA_OK) return st;
    for (int l = 0; l < (int)p.lanes.size(); ++l)
      for (int i = p.lanes[l].req_lo; i < p.lanes[l].req_hi; ++i) lane_of[p.order[i]] = l;
    return ROSA_OK;
  } catch (...) {
    return ROSA_E_NOMEM;
  }
}

rosa_status rosa_debug_time_conditioning(rosa_batch *b, const float *taus, int32_t n, float *out) {
  if (!b) return ROSA_E_INVALID;
  try {
    if (b->poisoned) return fail(b, ROSA_E_DEVICE, "handle is poisoned");
    if (!taus || !out || n < 1 || n > kMaxTau) return fail(b, ROSA_E_INVALID, "bad taus/out/n");
    hipError_t e = hipSetDevice(b->device);
    float *d_taus = (float *)((uint8_t *)b->d_plan + b->off_taus);
    if (e == hipSuccess) e = hipStreamSynchronize(b->stream);
    if (e == hipSuccess) e = hipMemcpy(d_taus, taus, n * 4, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = run_time_conditioning(b, d_taus, n, out);
    if (e != hipSuccess) return device_fail(b, e, "time conditioning");
    return ROSA_OK;
  } catch (...) {
    return fail(b, ROSA_E_DEVICE, "unexpected exception");
  }
}

rosa_status rosa_debug_attention(rosa_batch *b, const rosa_request *reqs, int32_t n, int32_t layer,
                                 const void *qkv, void *o) {
  if (!b) return ROSA_E_INVALID;
  try {
    if (b->poisoned) return fail(b, ROSA_E_DEVICE, "handle is poisoned");
    if (!qkv || !o || layer < 0 || layer >= b->dims.L) return fail(b, ROSA_E_INVALID, "bad qkv/o/layer");
    Plan p;
    std::string err;
    rosa_status st = build_plan(&b->cfg, &b->cap, reqs, n, false, b->bf16, 1, p, err);
    if (st != ROSA_OK) return fail(b, st, err);
    if (n == 0) return ROSA_OK;
    hipError_t e = hipSetDevice(b->device);
    if (e == hipSuccess) e = upload_plan(b, p, reqs, n);
    if (e == hipSuccess) e = run_attention(b, p, p.lanes[0], 0, layer, qkv, o, b->stream, 0);
    if (e != hipSuccess) return device_fail(b, e, "attention");
    return ROSA_OK;
  } catch (...) {
    return fail(b, ROSA_E_DEVICE, "unexpected exception");
  }
}

rosa_status rosa_attention_noalloc(const rosa_model_config *cfg, const rosa_request *reqs, int32_t n, int32_t layer,
                                   const void *qkv, void *o, void *hip_stream) {
  try {
    g_create_error.clear();
    if (!cfg) return fail(nullptr, ROSA_E_INVALID, "cfg is NULL");
    rosa_status st = check_config(cfg);
    if (st != ROSA_OK) return fail(nullptr, st, "model configuration not supported");
    if (n < 0 || (n > 0 && !reqs) || layer < 0 || layer >= cfg->n_layers)
      return fail(nullptr, ROSA_E_INVALID, "bad request count, request array or layer");
    if (n > kNaMaxRequests) return fail(nullptr, ROSA_E_CAPACITY, "more than 1024 requests");
    if (n == 0) return ROSA_OK;
    if (!qkv || !o || ((uintptr_t)qkv | (uintptr_t)o) & 15)
      return fail(nullptr, ROSA_E_INVALID, "qkv and o must be non-NULL and 16-byte aligned");
    // Capacity of exactly this request set (build_plan validates every request).
    rosa_capacity cap{};
    cap.max_requests = n;
    cap.max_steps = 1;
    int64_t sum_h = 0, sum_p = 0;
    for (int i = 0; i < n; ++i) {
      cap.max_horizon = std::max(cap.max_horizon, reqs[i].horizon);
      cap.max_steps = std::max(cap.max_steps, reqs[i].num_steps);
      sum_h += std::max(reqs[i].horizon, 0);
      sum_p += std::max(reqs[i].prefix_len, 0);
    }
    if (sum_h > INT32_MAX || cap.max_steps > kMaxSteps)
      return fail(nullptr, ROSA_E_INVALID, "sum of horizons or a step count out of range");
    cap.max_action_tokens = (int32_t)std::max<int64_t>(sum_h, 1);
    cap.max_horizon = std::max(cap.max_horizon, 1);
    cap.max_prefix_tokens = sum_p;
    const bool bf16 = cfg->dtype == ROSA_BF16;
    Plan p;
    std::string err;
    st = build_plan(cfg, &cap, reqs, n, false, bf16, 1, p, err, INT32_MAX, kNaMaxSlots);
    if (st != ROSA_OK) return fail(nullptr, st, err);
    const Plan::AttnSet &S0 = p.sets[0], &S1 = p.sets[1];
    const size_t n_items = S0.items.size() + S1.items.size(), n_groups = S0.groups.size() + S1.groups.size();
    if (n_items > (size_t)kNaMaxItems || n_groups > (size_t)kNaMaxSlots || p.attn_lists.size() > (size_t)kNaMaxItems)
      return fail(nullptr, ROSA_E_CAPACITY, "more than 4096 attention work items or launch blocks");

    // Host image of the plan regions, copied into the scratch in one transfer.
    std::vector<uint8_t> img(kNaOffMl, 0);
    ReqDesc *rd = reinterpret_cast<ReqDesc *>(img.data() + kNaOffReqs);
    for (int i = 0; i < n; ++i) {
      const rosa_request &r = reqs[p.order[i]];
      ReqDesc d{};
      d.pk = r.prefix_k; d.pv = r.prefix_v; d.noise = r.noise; d.actions = r.actions;
      d.P = r.prefix_len; d.H = r.horizon; d.K = r.num_steps; d.tok_off = p.tok_off[i]; d.orig = p.order[i];
      d.k0 = r.start_step; d.S = p.steps[i];
      rd[i] = d;
    }
    std::vector<AttnItem> all(S0.items);
    all.insert(all.end(), S1.items.begin(), S1.items.end());
    std::memcpy(img.data() + kNaOffItems, all.data(), all.size() * sizeof(AttnItem));
    std::memcpy(img.data() + kNaOffGroups, S0.groups.data(), S0.groups.size() * sizeof(AttnGroup));
    std::memcpy(img.data() + kNaOffGroups + S0.groups.size() * sizeof(AttnGroup), S1.groups.data(),
                S1.groups.size() * sizeof(AttnGroup));
    attn_order_items(all, p.attn_lists.data(), p.attn_next.data(), p.attn_lists.size(),
                     reinterpret_cast<AttnItem *>(img.data() + kNaOffLists));

    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    uint8_t *sp = nullptr;
    if (e == hipSuccess) e = noalloc_scratch(dev, &sp);
    const hipStream_t stream = (hipStream_t)hip_stream;
    const size_t used = kNaOffLists + p.attn_lists.size() * sizeof(AttnItem);
    if (e == hipSuccess) e = hipMemcpyAsync(sp, img.data(), used, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return device_fail(nullptr, e, "scratch address or plan upload");

    const Dims D = make_dims(cfg);
    const Plan::Lane &ln = p.lanes[0];
    const int v = attn_set_of(cfg, layer);
    const Plan::AttnSet &S = p.sets[v];
    AttnArgs a{};
    a.items = reinterpret_cast<const AttnItem *>(sp + kNaOffItems) + S.item_base;
    a.n_items = (int)S.items.size();
    if (bf16) {
      a.items = reinterpret_cast<const AttnItem *>(sp + kNaOffItems);
      a.ordered = reinterpret_cast<const AttnItem *>(sp + kNaOffLists) + ln.list_at[v][0];
      a.n_blocks = ln.list_blocks[v][0];
    }
    a.reqs = reinterpret_cast<const ReqDesc *>(sp + kNaOffReqs);
    a.layer = layer;
    a.qkv = qkv; a.ldqkv = D.qkv_dim; a.o = o; a.ldo = D.o_dim;
    a.nq = D.nq; a.nkv = D.nkv; a.hd = D.hd;
    a.part_o = sp + kNaOffO;
    a.part_ml = reinterpret_cast<float *>(sp + kNaOffMl);
    e = launch_attention(a, bf16, stream);
    if (e == hipSuccess && !S.groups.empty())
      e = launch_attn_merge(reinterpret_cast<const AttnGroup *>(sp + kNaOffGroups) + S.group_base, (int)S.groups.size(),
                            a.reqs, a.part_o, a.part_ml, o, D.o_dim, D.nq, D.nkv, D.hd, bf16, stream);
    return e == hipSuccess ? ROSA_OK : device_fail(nullptr, e, "attention launch");
  } catch (const std::bad_alloc &) {
    return fail(nullptr, ROSA_E_NOMEM, "host allocation failed");
  } catch (...) {
    return fail(nullptr, ROSA_E_DEVICE, "unexpected exception");
  }
}

rosa_status rosa_debug_gemm(rosa_batch *b, int32_t which, int32_t layer, const void *a, int32_t M, void *out,
                            const float *gate) {
  if (!b) return ROSA_E_INVALID;
  try {
    if (b->poisoned) return fail(b, ROSA_E_DEVICE, "handle is poisoned");
    const Dims &D = b->dims;
    if (which < 0 || which > 3 || layer < 0 || layer >= D.L || !a || !out || M < 0 ||
        M > b->cap.max_action_tokens || ((which == 1 || which == 3) && !gate))
      return fail(b, ROSA_E_INVALID, "bad gemm arguments");
    if (((uintptr_t)a | (uintptr_t)out | (uintptr_t)gate) & 15)
      return fail(b, ROSA_E_INVALID, "gemm operands must be 16-byte aligned");
    GemmArgs g{};
    g.a = a; g.M = M; g.out = out; g.gate = gate; g.rowmod = b->ident;
    g.part = b->gemm_part; g.part_floats = b->gemm_part_floats;
    switch (which) {
      case 0: g.lda = D.d; g.K = D.d; g.N = D.qkv_dim; g.epi = kEpiStore; g.ldo = D.qkv_dim;
              g.wt = (uint8_t *)b->wt_qkv + (size_t)layer * D.qkv_dim * D.d * b->esz; break;
      case 1: g.lda = D.o_dim; g.K = D.o_dim; g.N = D.d; g.epi = kEpiGatedResidual; g.ldo = D.d; g.gate_stride = D.d;
              g.wt = (uint8_t *)b->wt_o + (size_t)layer * D.d * D.o_dim * b->esz; break;
      case 2: g.lda = D.d; g.K = D.d; g.N = D.dff; g.epi = kEpiGelu; g.ldo = D.dff;
              g.wt = (uint8_t *)b->wt_up + (size_t)layer * D.dff * D.d * b->esz; break;
      default: g.lda = D.dff; g.K = D.dff; g.N = D.d; g.epi = kEpiGatedResidual; g.ldo = D.d; g.gate_stride = D.d;
               g.wt = (uint8_t *)b->wt_down + (size_t)layer * D.d * D.dff * b->esz; break;
    }
    const int cls = which == 0 ? kcGemmQKV : which == 1 ? kcGemmO : which == 2 ? kcGemmUp : kcGemmDown;
    hipError_t e = hipSetDevice(b->device);
    if (e == hipSuccess && b->bf16) {
      // The caller's row-major A, repacked kb32 into the workspace the step
      // loop uses for this operand; the output stays row-major.
      void *ws = which == 1 ? b->o : which == 3 ? b->g : b->u;
      e = launch_kb32_pack(a, M, g.K, g.lda, ws, b->kb_rows, b->stream);
      g.a = ws;
      g.a_rows = b->kb_rows;
    }
    if (e == hipSuccess) e = timed(b, cls, [&] { return launch_gemm(g, b->bf16, b->stream, b->gemm_cfg); });
    if (e != hipSuccess) return device_fail(b, e, "gemm");
    return ROSA_OK;
  } catch (...) {
    return fail(b, ROSA_E_DEVICE, "unexpected exception");
  }
}

rosa_status rosa_debug_set_lanes(rosa_batch *b, int32_t n) {
  if (!b) return ROSA_E_INVALID;
  if (n < 1 || n > kMaxLanes) return fail(b, ROSA_E_INVALID, "lane count out of range");
  b->lanes = n;
  return ROSA_OK;
}

rosa_status rosa_debug_gemm_config(rosa_batch *b, int32_t cfg, int32_t *n_configs) {
  if (!b) return ROSA_E_INVALID;
  if (n_configs) *n_configs = kGemmConfigs;
  if (cfg < -1 || cfg >= kGemmConfigs) return fail(b, ROSA_E_INVALID, "gemm configuration out of range");
  b->gemm_cfg = cfg;
  return ROSA_OK;
}

rosa_status rosa_debug_set_profiling(rosa_batch *b, int32_t enable) {
  if (!b) return ROSA_E_INVALID;
  try {
    if (b->poisoned) return fail(b, ROSA_E_DEVICE, "handle is poisoned");
    hipError_t e = harvest_profile(b);
    if (e != hipSuccess) return device_fail(b, e, "profile sync");
    for (int i = 0; i < kcCount; ++i) { b->prof_ms[i] = 0.0; b->prof_launches[i] = 0; }
    b->prof = enable != 0;
    return ROSA_OK;
  } catch (...) {
    return fail(b, ROSA_E_DEVICE, "unexpected exception");
  }
}

rosa_status rosa_debug_get_profile(rosa_batch *b, const char **names, int64_t *launches, double *total_ms,
                                   int32_t max, int32_t *n_out) {
  if (!b) return ROSA_E_INVALID;
  try {
    if (b->poisoned) return fail(b, ROSA_E_DEVICE, "handle is poisoned");
    hipError_t e = harvest_profile(b);
    if (e != hipSuccess) return device_fail(b, e, "profile sync");
    const int n = std::min<int>(max, kcCount);
    for (int i = 0; i < n; ++i) {
      if (names) names[i] = kClassNames[i];
      if (launches) launches[i] = b->prof_launches[i];
      if (total_ms) total_ms[i] = b->prof_ms[i];
    }
    if (n_out) *n_out = n;
    return ROSA_OK;
  } catch (...) {
    return fail(b, ROSA_E_DEVICE, "unexpected exception");
  }
}

}  // extern "C"
