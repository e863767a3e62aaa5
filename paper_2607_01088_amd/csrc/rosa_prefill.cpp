// C ABI of the prefix producer: a vision-language backbone over every job's
// embedded prefix tokens whose per-layer K and V projections are written to
// the job's prefix caches (the keys and values the action expert reads at the
// same layer, Sec. 2.2.1).  All jobs of a call run as one stacked batch of
// rows through the shared kernels: the plain RMSNorm is the modulated one with
// zero shift and scale, the residual GEMM epilogue takes a gate of ones, and
// the ragged attention runs with no cached prefix and each job's own tokens as
// its key sequence.  In the context form (for a head that cross-attends to the
// backbone's output) the backbone runs in full and one more GEMM projects its
// normalised output for every head layer.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/rosa_debug.h"
#include "../../include/rosa_prefill.h"
#include "rosa_internal.h"

using namespace rosa;

namespace {

enum PrefillClass {
  pcLoad = 0, pcNorm, pcGemmQKV, pcScatter, pcAttention, pcMerge, pcGemmO, pcGemmUp, pcGemmDown, pcRope, pcCount
};
const char *kPrefillClassNames[pcCount] = {"load",      "norm",       "gemm_qkv", "kv_scatter", "attention",
                                           "attn_merge", "gemm_o",    "gemm_up",  "gemm_down",  "rope"};

thread_local std::string g_prefill_create_error;

struct PrefillPlan {
  std::vector<PrefillJob> jobs;
  std::vector<ReqDesc> reqs;      // attention's view: no cached prefix, H = P tokens
  std::vector<int32_t> row_job;
  std::vector<AttnItem> items;
  std::vector<AttnGroup> groups;
  std::vector<int32_t> list, list_next;   // bf16 launch order (block item lists)
  int n_blocks = 0;
  int64_t M = 0;
  bool causal = false;                    // some job has a causal segment
};

}  // namespace

struct rosa_prefill {
  rosa_vlm_config cfg{};
  int L = 0, d = 0, nq = 0, nkv = 0, hd = 0, dff = 0, qkv_dim = 0, o_dim = 0;
  bool bf16 = true;
  size_t esz = 2;
  int device = 0;
  hipStream_t stream = nullptr;
  bool poisoned = false;
  int gemm_cfg = -1;                         // forced projection block configuration, -1: cost model
  std::string last_error;
  int32_t max_jobs = 0;
  int64_t max_tokens = 0;
  int max_items = 0;
  size_t max_list = 0;

  void *wt_qkv = nullptr, *wt_o = nullptr, *wt_up = nullptr, *wt_down = nullptr;  // [L][N][K]
  // Context form: every head layer's [K | V] projection side by side,
  // transposed ([Le * 2 n_kv hd][d]), and the projected rows [M][ctx_dim].
  bool context = false;
  int head_layers = 0, ctx_dim = 0;
  void *wt_ctx = nullptr, *ctx = nullptr;
  float *h = nullptr;
  void *u = nullptr, *qkv = nullptr, *o = nullptr, *g = nullptr;
  int ldg = 0;                               // fp32: row stride of g: d_mlp + 64, off a power of two
  int kb_rows = 0;                           // bf16: u, o, g kb32 with planes of max_tokens rows
  float *zeros = nullptr, *ones = nullptr;   // [d]: zero shift and scale, unit gate
  int32_t *rowmod = nullptr;                 // [max_tokens] zeros
  float *part_o = nullptr, *part_ml = nullptr;
  // Rotary position embedding of the queries and keys (rope_base > 0): the
  // (cos, sin) table for positions below max_tokens, refreshed per call.
  double rope_base = 0.0;
  float *rope_tab = nullptr;

  // plan region on the device + two pinned staging copies
  void *d_plan = nullptr;
  void *h_plan[2] = {nullptr, nullptr};
  hipEvent_t plan_copied[2] = {nullptr, nullptr};
  bool plan_pending[2] = {false, false};
  int plan_flip = 0;
  size_t off_jobs = 0, off_reqs = 0, off_rows = 0, off_items = 0, off_groups = 0, off_list = 0, plan_bytes = 0;

  std::vector<void *> allocations;

  bool prof = false;
  struct Pending { int cls; hipEvent_t a, b; };
  std::vector<Pending> pending;
  std::vector<hipEvent_t> free_events;
  int64_t prof_launches[pcCount] = {};
  double prof_ms[pcCount] = {};
};

namespace {

rosa_status pfail(rosa_prefill *h, rosa_status st, const std::string &msg) {
  if (h) h->last_error = msg;
  else g_prefill_create_error = msg;
  return st;
}

rosa_status pdevice_fail(rosa_prefill *h, hipError_t e, const char *what) {
  std::string msg = std::string(what) + ": " + hipGetErrorString(e);
  if (h) {
    h->poisoned = true;
    h->last_error = msg;
  } else {
    g_prefill_create_error = msg;
  }
  return ROSA_E_DEVICE;
}

template <typename T>
T *palloc(rosa_prefill *h, size_t count, hipError_t &e) {
  void *ptr = nullptr;
  if (e != hipSuccess) return nullptr;
  e = hipMalloc(&ptr, std::max<size_t>(count * sizeof(T), 256));
  if (e == hipSuccess) h->allocations.push_back(ptr);
  return (T *)ptr;
}

void pfree_all(rosa_prefill *h) {
  for (void *p : h->allocations) hipFree(p);
  h->allocations.clear();
  for (int i = 0; i < 2; ++i) {
    if (h->h_plan[i]) hipHostFree(h->h_plan[i]);
    if (h->plan_copied[i]) hipEventDestroy(h->plan_copied[i]);
    h->h_plan[i] = nullptr;
    h->plan_copied[i] = nullptr;
  }
  for (auto &p : h->pending) { hipEventDestroy(p.a); hipEventDestroy(p.b); }
  h->pending.clear();
  for (auto e : h->free_events) hipEventDestroy(e);
  h->free_events.clear();
}

template <typename F>
hipError_t ptimed(rosa_prefill *h, int cls, F &&launch) {
  if (!h->prof) return launch();
  hipEvent_t e0 = nullptr, e1 = nullptr;
  for (hipEvent_t *ev : {&e0, &e1}) {
    if (!h->free_events.empty()) { *ev = h->free_events.back(); h->free_events.pop_back(); }
    else if (hipEventCreate(ev) != hipSuccess) *ev = nullptr;
  }
  if (!e0 || !e1) return launch();
  hipEventRecord(e0, h->stream);
  const hipError_t err = launch();
  hipEventRecord(e1, h->stream);
  h->pending.push_back({cls, e0, e1});
  return err;
}

hipError_t pharvest(rosa_prefill *h) {
  hipError_t e = hipStreamSynchronize(h->stream);
  if (e != hipSuccess) return e;
  for (auto &p : h->pending) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      h->prof_ms[p.cls] += ms;
      h->prof_launches[p.cls] += 1;
    }
    h->free_events.push_back(p.a);
    h->free_events.push_back(p.b);
  }
  h->pending.clear();
  return hipSuccess;
}

rosa_status check_vlm_config(const rosa_vlm_config *c) {
  if (c->n_layers < 1 || c->d_model < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1 || c->head_dim < 1 ||
      c->d_mlp < 1 || !(c->rms_eps >= 0.f))
    return ROSA_E_INVALID;
  if (c->dtype != ROSA_BF16 && c->dtype != ROSA_FP32) return ROSA_E_INVALID;
  if (c->n_q_heads % c->n_kv_heads != 0) return ROSA_E_UNSUPPORTED;
  if (c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 128 && c->head_dim != 256)
    return ROSA_E_UNSUPPORTED;
  if (c->d_model % 128 || c->d_mlp % 128 || (c->n_q_heads * c->head_dim) % 128 || c->d_model > 4096)
    return ROSA_E_UNSUPPORTED;
  if (c->cache_form != ROSA_CACHE_PER_LAYER && c->cache_form != ROSA_CACHE_CONTEXT) return ROSA_E_INVALID;
  if (c->cache_form == ROSA_CACHE_CONTEXT && (c->head_layers < 1 || c->head_layers > 1024)) return ROSA_E_INVALID;
  if (!(c->rope_base == 0.f || (c->rope_base > 1.f && c->rope_base < 1e30f))) return ROSA_E_INVALID;
  return ROSA_OK;
}

// Query blocks of R query rows: 32-row groups, at most `per` per block.
int query_blocks(int R, int per) { return ((R + 31) / 32 + per - 1) / per; }

// Validation (all-or-nothing) and the plan: stacked rows in job order, the
// row -> job table, and the attention work items (per job and KV head, query
// blocks of the job's P * G query rows over the job's P keys; keys split over
// several items only while the launch has too few items to fill the GPU).
rosa_status build_prefill_plan(const rosa_prefill *h, const rosa_prefix_job *jobs, int n, PrefillPlan &p,
                               std::string &err) {
  if (n < 0) { err = "n < 0"; return ROSA_E_INVALID; }
  if (n > 0 && !jobs) { err = "jobs is NULL"; return ROSA_E_INVALID; }
  if (n > h->max_jobs) { err = "more jobs than max_jobs"; return ROSA_E_CAPACITY; }
  int64_t M = 0;
  for (int i = 0; i < n; ++i) {
    const rosa_prefix_job &j = jobs[i];
    char buf[160];
    if (j.prefix_len < 1 || j.causal_len < 0 || j.causal_len > j.prefix_len) {
      snprintf(buf, sizeof buf, "job %d: prefix_len=%d causal_len=%d out of range", i, j.prefix_len, j.causal_len);
      err = buf; return ROSA_E_INVALID;
    }
    if (!j.embeddings || !j.prefix_k || !j.prefix_v) {
      snprintf(buf, sizeof buf, "job %d: NULL pointer", i); err = buf; return ROSA_E_INVALID;
    }
    if (((uintptr_t)j.embeddings | (uintptr_t)j.prefix_k | (uintptr_t)j.prefix_v) & 15) {
      snprintf(buf, sizeof buf, "job %d: buffers must be 16-byte aligned", i); err = buf; return ROSA_E_INVALID;
    }
    M += j.prefix_len;
  }
  if (M > h->max_tokens) { err = "sum of prefix lengths above max_tokens"; return ROSA_E_CAPACITY; }
  p = PrefillPlan();
  p.M = M;
  p.jobs.resize(n);
  p.reqs.resize(n);
  p.row_job.resize(M);
  int64_t off = 0;
  for (int i = 0; i < n; ++i) {
    const rosa_prefix_job &j = jobs[i];
    p.jobs[i] = PrefillJob{j.embeddings, j.prefix_k, j.prefix_v, j.prefix_len, (int32_t)off};
    ReqDesc r{};
    r.pk = h->qkv; r.pv = h->qkv;   // never read: no cached prefix keys
    r.P = 0; r.H = j.prefix_len; r.K = 1; r.tok_off = (int32_t)off; r.orig = i; r.S = 1;
    p.reqs[i] = r;
    std::fill(p.row_job.begin() + off, p.row_job.begin() + off + j.prefix_len, i);
    off += j.prefix_len;
  }

  const int G = h->nq / h->nkv;
  const int gpb = 4 * attn_groups_per_wave(h->hd);
  int64_t total_qb = 0;
  for (int i = 0; i < n; ++i) {
    total_qb += (int64_t)h->nkv * query_blocks(jobs[i].prefix_len * G, gpb);
    if (jobs[i].causal_len > 0) p.causal = true;
  }
  const bool split = h->bf16 && total_qb > 0 && total_qb < kAttnSplitTarget;
  int slots = 0;
  std::vector<std::pair<int, int>> ranges;
  for (int i = 0; i < n; ++i) {
    const int P = jobs[i].prefix_len;
    // Tokens below b see each other; later tokens see the keys up to their own.
    const int b = P - jobs[i].causal_len;
    const int R = P * G, ngrp = (R + 31) / 32, nqb = query_blocks(R, gpb);
    int nsplit = 1, chunk = P;
    // A causal job's keys are not split: a split item could then hold no
    // visible key for some of its query rows.
    if (split && b == P) {
      const int want = (int)((kAttnSplitTarget + total_qb - 1) / total_qb);
      const int most = std::max(1, (P + kAttnMinSplitKeys - 1) / kAttnMinSplitKeys);
      nsplit = std::min(want, most);
      chunk = (P + nsplit - 1) / nsplit;
      chunk = (chunk + 63) / 64 * 64;
      nsplit = (P + chunk - 1) / chunk;
    }
    const int first = (int)p.items.size();
    for (int kvh = 0; kvh < h->nkv; ++kvh)
      for (int qb = 0; qb < nqb; ++qb) {
        const int q0 = 32 * (qb * ngrp / nqb);
        const int nq = std::min(R, 32 * ((qb + 1) * ngrp / nqb)) - q0;
        if (nsplit > 1) p.groups.push_back(AttnGroup{i, kvh, q0, nq, slots, nsplit, 0, 0});
        for (int c = 0; c < nsplit; ++c) {
          AttnItem it{};
          it.pk = h->qkv; it.pv = h->qkv; it.P = 0; it.tok_off = (int32_t)p.jobs[i].tok_off;
          it.req = i; it.kvh = kvh; it.q0 = q0; it.nq = nq;
          it.kbeg = c * chunk;
          it.kend = std::min(P, (c + 1) * chunk);
          it.slot = nsplit > 1 ? slots++ : -1;
          // Keys past the block's last token's limit are invisible to all its rows.
          it.causal_b = b;
          if (b < P) it.kend = std::min(it.kend, std::max(b, (q0 + nq - 1) / G + 1));
          p.items.push_back(it);
        }
      }
    ranges.push_back({first, (int)p.items.size()});
  }
  if (slots > kAttnMaxSlots || (int64_t)p.items.size() > h->max_items) {
    err = "internal: attention work items exceeded";
    return ROSA_E_CAPACITY;
  }
  if (h->bf16 && !p.items.empty()) p.n_blocks = attn_launch_order(p.items, ranges, p.list, p.list_next);
  if (p.list.size() > h->max_list) { err = "internal: attention launch order exceeded"; return ROSA_E_CAPACITY; }
  return ROSA_OK;
}

hipError_t upload_prefill_plan(rosa_prefill *h, const PrefillPlan &p) {
  const int slot = h->plan_flip;
  h->plan_flip ^= 1;
  if (h->plan_pending[slot]) {
    hipError_t e = hipEventSynchronize(h->plan_copied[slot]);
    if (e != hipSuccess) return e;
  }
  uint8_t *hp = (uint8_t *)h->h_plan[slot];
  std::memcpy(hp + h->off_jobs, p.jobs.data(), p.jobs.size() * sizeof(PrefillJob));
  std::memcpy(hp + h->off_reqs, p.reqs.data(), p.reqs.size() * sizeof(ReqDesc));
  std::memcpy(hp + h->off_rows, p.row_job.data(), p.row_job.size() * 4);
  std::memcpy(hp + h->off_items, p.items.data(), p.items.size() * sizeof(AttnItem));
  std::memcpy(hp + h->off_groups, p.groups.data(), p.groups.size() * sizeof(AttnGroup));
  attn_order_items(p.items, p.list.data(), p.list_next.data(), p.list.size(), (AttnItem *)(hp + h->off_list));
  const size_t used = h->off_list + p.list.size() * sizeof(AttnItem);
  hipError_t e = hipMemcpyAsync(h->d_plan, hp, used, hipMemcpyHostToDevice, h->stream);
  if (e != hipSuccess) return e;
  e = hipEventRecord(h->plan_copied[slot], h->stream);
  h->plan_pending[slot] = true;
  return e;
}

}  // namespace

extern "C" {

const char *rosa_prefill_last_error(const rosa_prefill *h) {
  return h ? h->last_error.c_str() : g_prefill_create_error.c_str();
}

rosa_status rosa_prefill_create(const rosa_vlm_config *cfg, const rosa_vlm_weights *w, int32_t max_jobs,
                                int64_t max_tokens, void *hip_stream, rosa_prefill **out) {
  try {
    g_prefill_create_error.clear();
    if (!out) return pfail(nullptr, ROSA_E_INVALID, "out is NULL");
    *out = nullptr;
    if (!cfg || !w) return pfail(nullptr, ROSA_E_INVALID, "NULL config or weights");
    rosa_status st = check_vlm_config(cfg);
    if (st != ROSA_OK) return pfail(nullptr, st, "backbone configuration not supported");
    if (max_jobs < 1 || max_tokens < 1 || max_tokens > INT32_MAX / 2)
      return pfail(nullptr, ROSA_E_INVALID, "bad max_jobs / max_tokens");
    // query rows of one job (tokens x query heads per KV head) are int32 in the plan and kernels
    if (max_tokens * (cfg->n_q_heads / cfg->n_kv_heads) > (int64_t(1) << 30))
      return pfail(nullptr, ROSA_E_UNSUPPORTED, "max_tokens x query heads per KV head above 2^30");
    if (!w->w_qkv || !w->w_o || !w->w_up || !w->w_down || (cfg->cache_form == ROSA_CACHE_CONTEXT && !w->w_ctx))
      return pfail(nullptr, ROSA_E_INVALID, "NULL weight pointer");

    rosa_prefill *h = new rosa_prefill();
    h->cfg = *cfg;
    h->L = cfg->n_layers; h->d = cfg->d_model; h->nq = cfg->n_q_heads; h->nkv = cfg->n_kv_heads;
    h->hd = cfg->head_dim; h->dff = cfg->d_mlp;
    h->qkv_dim = (h->nq + 2 * h->nkv) * h->hd;
    h->o_dim = h->nq * h->hd;
    h->bf16 = cfg->dtype == ROSA_BF16;
    h->esz = h->bf16 ? 2 : 4;
    h->stream = (hipStream_t)hip_stream;
    h->max_jobs = max_jobs;
    h->max_tokens = max_tokens;
    hipError_t e = hipGetDevice(&h->device);
    if (e != hipSuccess) { rosa_status s2 = pdevice_fail(nullptr, e, "hipGetDevice"); delete h; return s2; }

    const size_t L = h->L, d = h->d, T = (size_t)max_tokens, es = h->esz;
    h->wt_qkv = palloc<uint8_t>(h, L * h->qkv_dim * d * es, e);
    h->wt_o = palloc<uint8_t>(h, L * d * h->o_dim * es, e);
    h->wt_up = palloc<uint8_t>(h, L * h->dff * d * es, e);
    h->wt_down = palloc<uint8_t>(h, L * d * h->dff * es, e);
    h->context = cfg->cache_form == ROSA_CACHE_CONTEXT;
    if (h->context) {
      h->head_layers = cfg->head_layers;
      h->ctx_dim = h->head_layers * 2 * h->nkv * h->hd;
      h->wt_ctx = palloc<uint8_t>(h, (size_t)h->ctx_dim * d * es, e);
      h->ctx = palloc<uint8_t>(h, (size_t)max_tokens * h->ctx_dim * es, e);
    }
    h->h = palloc<float>(h, T * d, e);
    h->u = palloc<uint8_t>(h, T * d * es, e);
    h->qkv = palloc<uint8_t>(h, T * h->qkv_dim * es, e);
    h->o = palloc<uint8_t>(h, T * h->o_dim * es, e);
    h->ldg = h->dff + 64;
    h->kb_rows = h->bf16 ? (int)T : 0;
    h->g = palloc<uint8_t>(h, T * h->ldg * es, e);
    h->zeros = palloc<float>(h, d, e);
    h->ones = palloc<float>(h, d, e);
    h->rowmod = palloc<int32_t>(h, T, e);
    h->rope_base = cfg->rope_base;
    if (h->rope_base > 0.0) h->rope_tab = palloc<float>(h, T * h->hd, e);   // T positions x hd/2 (cos, sin)
    h->part_o = palloc<float>(h, (size_t)kAttnMaxSlots * kAttnQB * h->hd, e);
    h->part_ml = palloc<float>(h, (size_t)kAttnMaxSlots * kAttnQB * 2, e);

    const int G = h->nq / h->nkv;
    const int64_t qb_bound = (int64_t)h->nkv * (((int64_t)T * G + 127) / 128 + 2 * (int64_t)max_jobs);
    h->max_items = (int)(qb_bound + kAttnMaxSlots);
    h->max_list = 2 * (size_t)h->max_items + 8;
    auto align = [](size_t v) { return (v + 255) / 256 * 256; };
    h->off_jobs = 0;
    h->off_reqs = align(h->off_jobs + (size_t)max_jobs * sizeof(PrefillJob));
    h->off_rows = align(h->off_reqs + (size_t)max_jobs * sizeof(ReqDesc));
    h->off_items = align(h->off_rows + T * 4);
    h->off_groups = align(h->off_items + (size_t)h->max_items * sizeof(AttnItem));
    h->off_list = align(h->off_groups + (size_t)kAttnMaxSlots * sizeof(AttnGroup));
    h->plan_bytes = align(h->off_list + h->max_list * sizeof(AttnItem));
    h->d_plan = palloc<uint8_t>(h, h->plan_bytes, e);
    if (e != hipSuccess) {
      rosa_status s2 = e == hipErrorOutOfMemory ? pfail(nullptr, ROSA_E_NOMEM, "device allocation failed")
                                                 : pdevice_fail(nullptr, e, "hipMalloc");
      pfree_all(h); delete h; return s2;
    }
    for (int i = 0; i < 2 && e == hipSuccess; ++i) {
      e = hipHostMalloc(&h->h_plan[i], h->plan_bytes, hipHostMallocDefault);
      if (e == hipSuccess) e = hipEventCreateWithFlags(&h->plan_copied[i], hipEventDisableTiming);
    }
    if (e != hipSuccess) { rosa_status s2 = pfail(nullptr, ROSA_E_NOMEM, "pinned host allocation failed"); pfree_all(h); delete h; return s2; }

    if (e == hipSuccess) e = upload_gemm_weights(h->wt_qkv, w->w_qkv, h->L, h->d, h->qkv_dim, h->bf16);
    if (e == hipSuccess) e = upload_gemm_weights(h->wt_o, w->w_o, h->L, h->o_dim, h->d, h->bf16);
    if (e == hipSuccess) e = upload_gemm_weights(h->wt_up, w->w_up, h->L, h->d, h->dff, h->bf16);
    if (e == hipSuccess) e = upload_gemm_weights(h->wt_down, w->w_down, h->L, h->dff, h->d, h->bf16);
    if (e == hipSuccess && h->context) {
      // [Le][d][2 kv] -> [d][Le * 2 kv], then transposed like every projection
      const size_t kv2 = 2 * (size_t)h->nkv * h->hd;
      std::vector<float> cat(d * (size_t)h->ctx_dim);
      for (int l = 0; l < h->head_layers; ++l)
        for (size_t i = 0; i < d; ++i)
          std::memcpy(&cat[i * h->ctx_dim + l * kv2], w->w_ctx + ((size_t)l * d + i) * kv2, kv2 * 4);
      e = upload_gemm_weights(h->wt_ctx, cat.data(), 1, h->d, h->ctx_dim, h->bf16);
    }
    if (e == hipSuccess) {
      std::vector<float> one(d, 1.0f);
      e = hipMemcpy(h->ones, one.data(), d * 4, hipMemcpyHostToDevice);
    }
    if (e == hipSuccess) e = hipMemset(h->zeros, 0, d * 4);
    if (e == hipSuccess) e = hipMemset(h->rowmod, 0, T * 4);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) { rosa_status s2 = pdevice_fail(nullptr, e, "weight upload"); pfree_all(h); delete h; return s2; }
    *out = h;
    return ROSA_OK;
  } catch (const std::bad_alloc &) {
    return pfail(nullptr, ROSA_E_NOMEM, "host allocation failed");
  } catch (...) {
    return pfail(nullptr, ROSA_E_DEVICE, "unexpected exception");
  }
}

rosa_status rosa_prefill_run(rosa_prefill *h, const rosa_prefix_job *jobs, int32_t n) {
  if (!h) return ROSA_E_INVALID;
  try {
    h->last_error.clear();
    if (h->poisoned) return pfail(h, ROSA_E_DEVICE, "handle is poisoned by an earlier device error");
    PrefillPlan p;
    std::string err;
    rosa_status st = build_prefill_plan(h, jobs, n, p, err);
    if (st != ROSA_OK) return pfail(h, st, err);
    if (n == 0) return ROSA_OK;
    hipError_t e = hipSetDevice(h->device);
    if (e == hipSuccess) e = upload_prefill_plan(h, p);
    if (e != hipSuccess) return pdevice_fail(h, e, "plan upload");

    uint8_t *dp = (uint8_t *)h->d_plan;
    const PrefillJob *d_jobs = (const PrefillJob *)(dp + h->off_jobs);
    const ReqDesc *d_reqs = (const ReqDesc *)(dp + h->off_reqs);
    const int32_t *d_rows = (const int32_t *)(dp + h->off_rows);
    const AttnItem *d_items = (const AttnItem *)(dp + h->off_items);
    const AttnGroup *d_groups = (const AttnGroup *)(dp + h->off_groups);
    const AttnItem *d_list = (const AttnItem *)(dp + h->off_list);
    const int M = (int)p.M;
    const size_t es = h->esz;
    const hipStream_t s = h->stream;

    e = ptimed(h, pcLoad, [&] { return launch_prefill_load(d_jobs, d_rows, M, h->d, h->bf16, h->h, s); });
    if (e == hipSuccess && h->rope_tab) {
      int max_p = 0;
      for (int i = 0; i < n; ++i) max_p = std::max(max_p, jobs[i].prefix_len);
      e = ptimed(h, pcRope, [&] { return launch_prefill_rope_table(h->rope_tab, max_p, h->hd, h->rope_base, s); });
    }
    for (int l = 0; l < h->L && e == hipSuccess; ++l) {
      e = ptimed(h, pcNorm, [&] {
        return launch_modnorm(h->h, M, h->d, h->cfg.rms_eps, h->zeros, 0, 0, 0, h->rowmod, h->u, h->bf16, s,
                              h->kb_rows);
      });
      if (e != hipSuccess) break;
      GemmArgs gq{};
      gq.a = h->u; gq.lda = h->d; gq.a_rows = h->kb_rows; gq.wt = (uint8_t *)h->wt_qkv + (size_t)l * h->qkv_dim * h->d * es;
      gq.M = M; gq.N = h->qkv_dim; gq.K = h->d; gq.epi = kEpiStore; gq.out = h->qkv; gq.ldo = h->qkv_dim;
      e = ptimed(h, pcGemmQKV, [&] { return launch_gemm(gq, h->bf16, s, h->gemm_cfg); });
      if (e == hipSuccess && h->rope_tab)
        e = ptimed(h, pcRope, [&] {
          return launch_prefill_rope(d_jobs, d_rows, M, h->qkv, h->qkv_dim, h->nq + h->nkv, h->hd, h->bf16,
                                     h->rope_tab, s);
        });
      if (e != hipSuccess) break;
      if (!h->context) {
        e = ptimed(h, pcScatter, [&] {
          return launch_prefill_kv_scatter(d_jobs, d_rows, M, h->qkv, h->qkv_dim, h->nq, h->nkv, h->hd, es, l, s);
        });
        // The last layer's attention and MLP feed nothing this call returns:
        // its caches are complete once its K and V are stored.
        if (e != hipSuccess || l == h->L - 1) break;
      }
      AttnArgs a{};
      a.items = d_items; a.n_items = (int)p.items.size();
      a.ordered = d_list; a.n_blocks = p.n_blocks;
      a.reqs = d_reqs; a.layer = 0;
      a.qkv = h->qkv; a.ldqkv = h->qkv_dim; a.o = h->o; a.ldo = h->o_dim; a.o_rows = h->kb_rows;
      a.nq = h->nq; a.nkv = h->nkv; a.hd = h->hd;
      a.part_o = h->part_o; a.part_ml = h->part_ml;
      a.causal = p.causal ? 1 : 0;
      e = ptimed(h, pcAttention, [&] { return launch_attention(a, h->bf16, s); });
      if (e == hipSuccess && !p.groups.empty())
        e = ptimed(h, pcMerge, [&] {
          return launch_attn_merge(d_groups, (int)p.groups.size(), d_reqs, h->part_o, h->part_ml, h->o, h->o_dim,
                                   h->nq, h->nkv, h->hd, h->bf16, s, h->kb_rows);
        });
      if (e != hipSuccess) break;
      GemmArgs go{};
      go.a = h->o; go.lda = h->o_dim; go.a_rows = h->kb_rows; go.wt = (uint8_t *)h->wt_o + (size_t)l * h->d * h->o_dim * es;
      go.M = M; go.N = h->d; go.K = h->o_dim; go.epi = kEpiGatedResidual; go.out = h->h; go.ldo = h->d;
      go.gate = h->ones; go.gate_stride = 0; go.rowmod = h->rowmod;
      e = ptimed(h, pcGemmO, [&] { return launch_gemm(go, h->bf16, s, h->gemm_cfg); });
      if (e != hipSuccess) break;
      e = ptimed(h, pcNorm, [&] {
        return launch_modnorm(h->h, M, h->d, h->cfg.rms_eps, h->zeros, 0, 0, 0, h->rowmod, h->u, h->bf16, s,
                              h->kb_rows);
      });
      if (e != hipSuccess) break;
      GemmArgs gu{};
      gu.a = h->u; gu.lda = h->d; gu.a_rows = h->kb_rows; gu.out_rows = h->kb_rows; gu.wt = (uint8_t *)h->wt_up + (size_t)l * h->dff * h->d * es;
      gu.M = M; gu.N = h->dff; gu.K = h->d; gu.epi = kEpiGelu; gu.out = h->g; gu.ldo = h->ldg;
      e = ptimed(h, pcGemmUp, [&] { return launch_gemm(gu, h->bf16, s, h->gemm_cfg); });
      if (e != hipSuccess) break;
      GemmArgs gd{};
      gd.a = h->g; gd.lda = h->ldg; gd.a_rows = h->kb_rows; gd.wt = (uint8_t *)h->wt_down + (size_t)l * h->d * h->dff * es;
      gd.M = M; gd.N = h->d; gd.K = h->dff; gd.epi = kEpiGatedResidual; gd.out = h->h; gd.ldo = h->d;
      gd.gate = h->ones; gd.gate_stride = 0; gd.rowmod = h->rowmod;
      e = ptimed(h, pcGemmDown, [&] { return launch_gemm(gd, h->bf16, s, h->gemm_cfg); });
    }
    if (h->context && e == hipSuccess) {
      // Final RMSNorm, one projection for every head layer, then each layer's
      // [K | V] column block into the caches.
      e = ptimed(h, pcNorm, [&] {
        return launch_modnorm(h->h, M, h->d, h->cfg.rms_eps, h->zeros, 0, 0, 0, h->rowmod, h->u, h->bf16, s,
                              h->kb_rows);
      });
      GemmArgs gc{};
      gc.a = h->u; gc.lda = h->d; gc.a_rows = h->kb_rows; gc.wt = h->wt_ctx;
      gc.M = M; gc.N = h->ctx_dim; gc.K = h->d; gc.epi = kEpiStore; gc.out = h->ctx; gc.ldo = h->ctx_dim;
      if (e == hipSuccess) e = ptimed(h, pcGemmQKV, [&] { return launch_gemm(gc, h->bf16, s, h->gemm_cfg); });
      const size_t kv2_bytes = 2 * (size_t)h->nkv * h->hd * es;
      for (int l = 0; l < h->head_layers && e == hipSuccess; ++l)
        e = ptimed(h, pcScatter, [&] {
          return launch_prefill_kv_scatter(d_jobs, d_rows, M, (const uint8_t *)h->ctx + l * kv2_bytes, h->ctx_dim, 0,
                                           h->nkv, h->hd, es, l, s);
        });
    }
    if (e != hipSuccess) return pdevice_fail(h, e, "kernel launch");
    return ROSA_OK;
  } catch (const std::bad_alloc &) {
    return pfail(h, ROSA_E_NOMEM, "host allocation failed");
  } catch (...) {
    return pfail(h, ROSA_E_DEVICE, "unexpected exception");
  }
}

void rosa_prefill_destroy(rosa_prefill *h) {
  if (!h) return;
  try {
    hipSetDevice(h->device);
    hipStreamSynchronize(h->stream);
    pfree_all(h);
  } catch (...) {
  }
  delete h;
}

rosa_status rosa_debug_prefill_set_profiling(rosa_prefill *h, int32_t enable) {
  if (!h) return ROSA_E_INVALID;
  try {
    if (h->poisoned) return pfail(h, ROSA_E_DEVICE, "handle is poisoned");
    hipError_t e = pharvest(h);
    if (e != hipSuccess) return pdevice_fail(h, e, "profile sync");
    for (int i = 0; i < pcCount; ++i) { h->prof_ms[i] = 0.0; h->prof_launches[i] = 0; }
    h->prof = enable != 0;
    return ROSA_OK;
  } catch (...) {
    return pfail(h, ROSA_E_DEVICE, "unexpected exception");
  }
}

rosa_status rosa_debug_prefill_gemm_config(rosa_prefill *h, int32_t cfg, int32_t *n_configs) {
  if (!h) return ROSA_E_INVALID;
  if (n_configs) *n_configs = kGemmConfigs;
  if (cfg < -1 || cfg >= kGemmConfigs) return pfail(h, ROSA_E_INVALID, "gemm configuration out of range");
  h->gemm_cfg = cfg;
  return ROSA_OK;
}

rosa_status rosa_debug_prefill_get_profile(rosa_prefill *h, const char **names, int64_t *launches,
                                           double *total_ms, int32_t max, int32_t *n_out) {
  if (!h) return ROSA_E_INVALID;
  try {
    if (h->poisoned) return pfail(h, ROSA_E_DEVICE, "handle is poisoned");
    hipError_t e = pharvest(h);
    if (e != hipSuccess) return pdevice_fail(h, e, "profile sync");
    const int n = std::max(0, std::min<int>(max, pcCount));
    for (int i = 0; i < n; ++i) {
      if (names) names[i] = kPrefillClassNames[i];
      if (launches) launches[i] = h->prof_launches[i];
      if (total_ms) total_ms[i] = h->prof_ms[i];
    }
    if (n_out) *n_out = n;
    return ROSA_OK;
  } catch (...) {
    return pfail(h, ROSA_E_DEVICE, "unexpected exception");
  }
}

}  // extern "C"
