// Internal structures shared by the host planner and the kernels' launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>
#include <vector>

namespace rosa {

// Per-request descriptor on the device (64 bytes), in plan order (K descending).
struct ReqDesc {
  const void *pk;        // prefix K, [L][P][n_kv][hd]
  const void *pv;        // prefix V, same layout
  const float *noise;    // [H][A]
  float *actions;        // [H][A]
  int32_t P, H, K, tok_off;
  int32_t orig;
  int32_t k0;            // Euler steps done before this call (x starts from actions if > 0)
  int32_t S;             // steps this call runs; the state goes to actions after step S-1
  int32_t pad0;
};
static_assert(sizeof(ReqDesc) == 64, "ReqDesc is 64 bytes");

// One attention work item: query rows [q0, q0 + nq) (nq <= kAttnQB) of KV head
// `kvh` of request `req`, over keys [kbeg, kend) of the request's key sequence
// (prefix keys first, then its action keys).  Query row q of a KV head is
// action token q / G, query head kvh * G + q % G (G query heads per KV head).
// slot >= 0: write unnormalized partial results to partial slot `slot`;
// slot < 0: write o directly.
// The request's prefix pointers, prefix length and first stacked row are
// copied in, so a block needs one load to start its copies.
struct AttnItem {
  const void *pk, *pv;   // the request's prefix K and V, [L][P][n_kv][hd]
  int32_t req, kvh, q0, nq, kbeg, kend, slot;
  int32_t P, tok_off;
  int32_t next;          // launch lists: the block's next entry, -1 after its last
  // Causal launches (AttnArgs::causal) only: key j is visible to the query
  // rows of token t (counted from the request's first token) iff
  // j < max(causal_b, t + 1), i.e. tokens below causal_b see each other and
  // every later token sees the keys up to itself.
  int32_t causal_b;
  int32_t pad2;
};
static_assert(sizeof(AttnItem) == 64, "AttnItem is 64 bytes");

// A query block whose keys were split over n items (partial slots first_slot
// .. first_slot + n - 1).
struct AttnGroup {
  int32_t req, kvh, q0, nq, first_slot, n, pad0, pad1;
};
static_assert(sizeof(AttnGroup) == 32, "AttnGroup is 32 bytes");

constexpr int kAttnQB = 256;       // most query rows per attention work item (4 waves x 2 x 32)
// 32-row query groups per wave of the bf16 attention kernel: two where Q^T and
// O^T of both fit half the register file (two waves share a SIMD), one from
// head_dim 128.  Work items hold at most 128 x this rows.
constexpr int attn_groups_per_wave(int hd) { return hd <= 64 ? 2 : 1; }
// Keys of a query block are split over several work items only while a
// launch has fewer than kAttnSplitTarget items; a split item holds at least
// kAttnMinSplitKeys keys; at most kAttnMaxSlots partial-result slots per launch.
constexpr int kAttnSplitTarget = 256;
// Persistent blocks of the bf16 attention kernel per launch: two per compute
// unit of a 256-CU MI355X.
constexpr int kAttnBlocks = 512;
constexpr int kAttnMinSplitKeys = 64;
constexpr int kAttnMaxSlots = 2 * kAttnSplitTarget;
constexpr int kMaxTau = 128;       // distinct flow times per call
constexpr int kMaxSteps = 64;

// Dimensions a launch needs.
struct Dims {
  int L, d, nq, nkv, hd, dff, A, dt, qkv_dim, o_dim, mod_stride;
  float eps;
};

enum Epilogue : int {
  kEpiStore = 0,          // out = acc                      (activation dtype)
  kEpiGelu = 1,           // out = gelu_tanh(acc)           (activation dtype)
  kEpiGatedResidual = 2,  // h += gate[rowmod[m]][n] * acc  (fp32)
  kEpiPartial = 3,        // out = acc (fp32): one K slice of a split product
};

// One job of the prefix producer on the device (32 bytes): its embedded
// tokens [P][d], its caches [L][P][n_kv][hd] (activation dtype) and its first
// stacked row.
struct PrefillJob {
  const void *emb;
  void *k, *v;
  int32_t P, tok_off;
};
static_assert(sizeof(PrefillJob) == 32, "PrefillJob is 32 bytes");

// ---------------------------------------------------------------- launchers
// All return hipGetLastError() of the launch.  `bf16` selects the activation
// and weight dtype (true: bf16, false: fp32).

// Time conditioning.
hipError_t launch_time_embedding(const float *taus, int n_tau, int dt, float *emb, hipStream_t s);
// Y[n][N] = act(X[n][K] W[K][N] + b); act: 0 none, 1 SiLU.  W row-major [K][N].
// ws: workspace of small_gemv_workspace_floats(N) floats (K-slice partials).
constexpr int kGemvMaxSlices = 8;
size_t small_gemv_workspace_floats(int N);
hipError_t launch_small_gemv(const float *X, int n, int K, const void *W, bool w_bf16, const float *b,
                             int N, int act, float *Y, float *ws, hipStream_t s);

// Row kernels.
hipError_t launch_setup_rows(const ReqDesc *reqs, int n_req, const int32_t *tau_idx, int max_steps,
                             int A, int32_t *row_req, int32_t *rowmod, int M0, float *x, hipStream_t s);
hipError_t launch_in_proj(const float *x, int M, int A, const float *w_in, const float *b_in, int d,
                          float *h, hipStream_t s);
// u: bf16 mode with u_rows > 0: kb32 planes of u_rows rows; else row-major [M][d].
hipError_t launch_modnorm(const float *h, int M, int d, float eps, const float *modtab, int mod_stride,
                          int shift_off, int scale_off, const int32_t *rowmod, void *u, bool bf16,
                          hipStream_t s, int u_rows = 0);
// bf16 row-major [M][K] (row stride lda) -> kb32 planes of R rows.
hipError_t launch_kb32_pack(const void *src, int M, int K, int lda, void *dst, int R, hipStream_t s);
hipError_t launch_final_euler(const float *h, int M, int d, float eps, const float *modtab,
                              int mod_stride, int shift_off, int scale_off, const int32_t *rowmod,
                              const float *w_out, const float *b_out, int A, const int32_t *row_req,
                              const ReqDesc *reqs, int step, float *x, int row0, hipStream_t s);

// bf16 mode: v = u W_out + b_out on final-normalized rows u (bf16 [M][d], or kb32
// planes of u_rows rows when u_rows > 0), Euler step
// x += v / K per row's request, actions written on its last step.  wt = W_out^T bf16 [A][d].
// u, row_req and x point at the first of the M rows, which is stacked row row0.
hipError_t launch_out_proj_euler(const __bf16 *u, int M, int d, const __bf16 *wt, const float *b_out, int A,
                                 const int32_t *row_req, const ReqDesc *reqs, int step, float *x, int row0,
                                 hipStream_t s, int u_rows = 0);

// K-blocked layout of a bf16 GEMM operand ("kb32"): element (m, k) of a
// matrix with planes of R rows at ((k / 32) * R + m) * 32 + k % 32, i.e. the
// matrix cut into 32-wide column blocks, each stored as R contiguous 64-byte
// rows.  A copy of 16 (or 8 twice) consecutive rows of one block is then 1 KB
// of contiguous memory.  kb32_offset gives the element offset.
__host__ __device__ inline size_t kb32_offset(size_t R, size_t m, size_t k) { return ((k >> 5) * R + m) * 32 + (k & 31); }

// GEMM: C[M][N] = A[M][K] * W^T.  fp32 mode: A row-major (lda), Wt [N][K]
// (K contiguous).  bf16 mode: A kb32 with planes of a_rows rows, Wt kb32 with
// planes of N rows ([K/32][N][32]).
struct GemmArgs {
  const void *a; int lda; int a_rows;
  const void *wt;            // [N][K]
  int M, N, K;
  int epi;
  void *out; int ldo;        // kEpiStore / kEpiGelu: activation dtype; kEpiGatedResidual: fp32 h
  int out_rows;              // bf16 kEpiStore / kEpiGelu: 0 row-major (ldo), else kb32 planes of out_rows rows
  const float *gate; int gate_stride; const int32_t *rowmod;  // gate = gate[rowmod[m]*gate_stride + n]
  // Optional fp32 workspace of part_floats floats.  When a launch would have
  // fewer than kSplitMinTiles tiles (few rows), K is split over up to
  // kSplitMax blocks per tile: each writes its slice's product here, and a
  // second kernel sums the slices in order and applies the epilogue.
  float *part; size_t part_floats;
  // Deferred modulated RMSNorm (bf16, unsplit launches only).  A
  // kEpiGatedResidual launch with dt set also leaves, for the rows it
  // updates, t = bf16(h (1 + scale)) (scale at dscale[rowmod[m] * gate_stride
  // + n]; kb32 planes of dt_rows rows) and the sum of squares of each row of h
  // over every 32-column block, dss[m * (N / 32) + n / 32].  A kEpiStore or
  // kEpiGelu launch with css set takes such a t as A and completes the norm
  // in its epilogue: acc / sqrt(ss_m / cd + ceps) + cshift[rowmod[m] *
  // cshift_stride + n], ss_m the sum of css[m * cparts .. + cparts) (cparts a
  // multiple of 8, at most 32) and
  // cshift the norm's shift multiplied by this launch's W, per modulation row.
  void *dt; int dt_rows; float *dss; const float *dscale;
  const float *css; int cparts, cd; float ceps; const float *cshift; int cshift_stride;
};
constexpr int kSplitMinTiles = 64;
constexpr int kSplitMinTilesNorm = 128;
constexpr int kSplitMax = 8;
// The modulated RMSNorm that consumes the rows a gated-residual projection
// has just updated: u[m] = RMSNorm(h[m]) (1 + scale) + shift, scale and shift
// at modtab[rowmod[m] * mod_stride + scale_off / shift_off + n] (rowmod: the
// projection's own).  u is bf16: kb32 planes of u_rows rows, or row-major
// [M][N] when u_rows = 0.
struct NormArgs {
  const float *modtab; int mod_stride; int shift_off; int scale_off; float eps;
  void *u; int u_rows;
};
// force_cfg < 0: block configuration chosen by the cost model.  With
// then_norm (kEpiGatedResidual, bf16, N <= kFusedNormMax), a product whose K
// is split has the norm fused into the kernel that sums its slices; *normed
// tells the caller whether that happened (else it launches the norm itself).
constexpr int kFusedNormMax = 1024;
// A gated-residual launch with dt set that is not split this way runs
// unsplit with the deferred norm's outputs (*deferred = true).
hipError_t launch_gemm(const GemmArgs &g, bool bf16, hipStream_t s, int force_cfg = -1,
                       const NormArgs *then_norm = nullptr, bool *normed = nullptr, bool *deferred = nullptr);
bool gemm_defers(const GemmArgs &g, int force_cfg, const NormArgs *then_norm);
// The shift halves of a deferred norm's products: for layer l < L, modulation
// row r < n_mod and column n, S[(l * n_mod + r) * (Nq + Nu) + n] = sum_k
// modtab[r * mod_stride + l * layer_stride + q_off + k] * Wq_l[k][n] for n < Nq,
// and the same with u_off and Wu_l for the Nu columns after them (Wq, Wu:
// bf16 kb32 [K/32][N][32] per layer, K = d).
hipError_t launch_shift_proj(const float *modtab, int mod_stride, int n_mod, int L, int layer_stride, int q_off,
                             int u_off, int d, const void *wq, int Nq, const void *wu, int Nu, float *S,
                             hipStream_t s);
// bf16 GEMM with a given block configuration (an index into the launcher's
// table of kGemmConfigs tiles, from 384 x 128 down to 64 x 32).
constexpr int kGemmConfigs = 13;
hipError_t launch_gemm_cfg(const GemmArgs &g, int cfg, hipStream_t s);
int gemm_pick_config(int M, int N, int K, int epi, int n_cu);

// Prefix producer rows.  row_job[row]: the job of stacked row `row`.
// h[row] = the job's embedding row (bf16 or fp32 in, fp32 out), d % 4 == 0.
hipError_t launch_prefill_load(const PrefillJob *jobs, const int32_t *row_job, int64_t M, int d, bool bf16_in,
                               float *h, hipStream_t s);
// Rotary position table [n_pos][head_dim / 2] of (cos, sin) pairs (fp32
// values computed in double): angle p * base^(-2 i / head_dim).
hipError_t launch_prefill_rope_table(float *tab, int n_pos, int head_dim, double base, hipStream_t s);
// Rotary position embedding, in place, of the first nheads heads of every
// stacked QKV row (queries, then keys) at the row's position within its job.
hipError_t launch_prefill_rope(const PrefillJob *jobs, const int32_t *row_job, int64_t M, void *qkv, int ldqkv,
                               int nheads, int head_dim, bool bf16_mode, const float *tab, hipStream_t s);
// Layer `layer`'s K and V column blocks of the stacked QKV rows into each job's
// caches; esz: bytes per element.
hipError_t launch_prefill_kv_scatter(const PrefillJob *jobs, const int32_t *row_job, int64_t M, const void *qkv,
                                     int ldqkv, int nq, int nkv, int hd, size_t esz, int layer, hipStream_t s);

// Attention of one layer.
struct AttnArgs {
  const AttnItem *items; int n_items;
  // bf16: the persistent blocks' item lists.  Block b runs ordered[b], then
  // the entry its `next` names, and so on until next is -1 (an idle block's
  // entry has nq 0); n_blocks blocks.  items and n_items are then unused.
  const AttnItem *ordered; int n_blocks;
  const ReqDesc *reqs;
  int layer;
  const void *qkv; int ldqkv;      // q at column g*hd, k_a at (nq+j)*hd, v_a at (nq+nkv+j)*hd
  void *o; int ldo;                // o at column g*hd
  int o_rows;                      // bf16: 0 row-major (ldo), else kb32 planes of o_rows rows
  int nq, nkv, hd;
  void *part_o;                    // [slot][kAttnQB][hd] bf16 (unnormalised O of split items)
  float *part_ml;                  // [slot][kAttnQB][2] fp32 (running max in log2 units, sum)
  // 1: every item's causal_b masks keys per query token (the prefix
  // producer's causal segments); such items are never key-split.
  int causal;
};
hipError_t launch_attention(const AttnArgs &a, bool bf16, hipStream_t s);
// Host: XCD-balanced item lists of persistent blocks for the items of the
// given requests (contiguous item ranges): appends entries to out (item
// index; entries 0 .. n_blocks-1 are the blocks' first items, -1: idle) and
// next (the index within this table of the block's next entry, -1 after its
// last); returns n_blocks.
int attn_launch_order(const std::vector<AttnItem> &items, const std::vector<std::pair<int, int>> &ranges,
                      std::vector<int32_t> &out, std::vector<int32_t> &next);
// Host: round-to-nearest-even fp32 -> bf16 bits (NaN stays a quiet NaN).
uint16_t f32_to_bf16_rne(float f);
// Host: upload L stacked [K][N] fp32 matrices as [L][N][K] (K contiguous), in
// bf16 or fp32; synchronous.
hipError_t upload_weights_transposed(void *dst, const float *src, int L, int K, int N, bool bf16);
// Host: the projection weights of the bf16 GEMM: L stacked [K][N] fp32
// matrices as bf16 kb32 [L][K/32][N][32]; synchronous.
hipError_t upload_weights_kb32(void *dst, const float *src, int L, int K, int N);
// The projection weights in the form launch_gemm expects for the mode.
inline hipError_t upload_gemm_weights(void *dst, const float *src, int L, int K, int N, bool bf16) {
  return bf16 ? upload_weights_kb32(dst, src, L, K, N) : upload_weights_transposed(dst, src, L, K, N, false);
}
// Host: the block lists as item records (an idle block gets an item with
// nq = 0), each with its `next` link, written to dst.
void attn_order_items(const std::vector<AttnItem> &items, const int32_t *order, const int32_t *next, size_t n,
                      AttnItem *dst);
hipError_t launch_attn_merge(const AttnGroup *groups, int n_groups, const ReqDesc *reqs,
                             const void *part_o, const float *part_ml, void *o, int ldo, int nq,
                             int nkv, int hd, bool bf16, hipStream_t s, int o_rows = 0);

}  // namespace rosa
