/*
 * rosa_debug.h - component entry points of the rosa library, for tests and
 * for per-kernel timing.  Same conventions as rosa.h: pure C, noexcept, status
 * returns, asynchronous on the handle's stream unless stated otherwise.
 */
#ifndef ROSA_DEBUG_H_
#define ROSA_DEBUG_H_

#include "rosa.h"
#include "rosa_prefill.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Host-only planning of a request set (no GPU needed, nothing enqueued): runs
 * the same validation and batch plan as rosa_generate_actions.
 *   order[n]      : plan position -> caller index (requests sorted by K
 *                   descending, stable), so the requests active at step k are a
 *                   prefix of the plan
 *   tok_off[n]    : first stacked action-token row of each request, by caller index
 *   m_k[cap->max_steps] : stacked action tokens active at step k (0 past the last step)
 *   counts[4]     : distinct flow times, attention work items, attention query
 *                   groups, query groups whose keys are split over several items
 * Any output pointer may be NULL.  Returns the status rosa_generate_actions
 * would return for this set (ROSA_E_DEVICE never). */
rosa_status rosa_debug_plan(const rosa_model_config *cfg, const rosa_capacity *cap,
                            const rosa_request *reqs, int32_t n, int32_t *order,
                            int32_t *tok_off, int32_t *m_k, int32_t *counts);

/* Host-only lane assignment of a request set (no GPU needed, nothing
 * enqueued): the lanes a bf16 call would split this set into when `lanes`
 * lanes are configured (rosa_debug_set_lanes), with the same rule as
 * rosa_generate_actions (at most n / 64 lanes).  lane_of[n] (by caller index)
 * receives each request's lane in [0, lanes).  Returns the status
 * rosa_generate_actions would return for this set. */
rosa_status rosa_debug_plan_lanes(const rosa_model_config *cfg, const rosa_capacity *cap,
                                  const rosa_request *reqs, int32_t n, int32_t lanes, int32_t *lane_of);

/* Host-only attention launch lists (bf16 configs; no GPU needed, nothing
 * enqueued): the persistent-block lists of the first attention launch of a
 * one-lane call over this set (step 0, every request active, the first
 * layer's attention set).
 *   n_blocks      : blocks launched; block b starts at entry b
 *   n_entries     : table entries (>= n_blocks)
 *   item_of[e]    : plan attention item of entry e (-1: an idle block)
 *   next[e]       : the same block's next entry, -1 after its last
 *   item_cost[i]  : 32-key steps of plan attention item i (counts[1] items of
 *                   rosa_debug_plan, first attention set)
 * item_of / next hold max_entries; ROSA_E_CAPACITY (counts still written)
 * when the table is longer.  Any array pointer may be NULL.  ROSA_E_UNSUPPORTED
 * for fp32 configs. */
rosa_status rosa_debug_attn_lists(const rosa_model_config *cfg, const rosa_capacity *cap,
                                  const rosa_request *reqs, int32_t n, int32_t max_entries,
                                  int32_t *n_blocks, int32_t *n_entries, int32_t *item_of,
                                  int32_t *next, int32_t *item_cost);

/* Attainable dense bf16 MFMA throughput of GPU `device`: times a kernel that
 * issues nothing but back-to-back v_mfma_f32_32x32x16_bf16 (eight
 * independent accumulators per wave, two waves per SIMD on every CU) and
 * writes the rate in TFLOP/s to *tflops (the clock the chip holds under that
 * load sets it, not the boost clock of the published peak).  Synchronous,
 * about 10 ms; allocates and frees a small buffer and a stream.
 * ROSA_E_DEVICE on any HIP error. */
rosa_status rosa_debug_mfma_peak(int32_t device, double *tflops);

/* Time conditioning alone: for n flow times taus (HOST fp32), write the
 * modulation table rows to out (DEVICE fp32 [n][L*6d + 2d]): per layer l the
 * six d-wide vectors [shift_a|scale_a|gate_a|shift_m|scale_m|gate_m] at offset
 * l*6d, then the final [shift|scale] at L*6d.  n <= 128. */
rosa_status rosa_debug_time_conditioning(rosa_batch *b, const float *taus, int32_t n, float *out);

/* Attention of one layer alone.  qkv: DEVICE [sum H][(n_q+2n_kv)*head_dim] in
 * the model dtype, the fused projection of each request's action tokens, rows
 * stacked in the caller's request order; o: DEVICE [sum H][n_q*head_dim] model
 * dtype, written.  Keys and values are the requests' prefix (layer `layer`)
 * followed by the k/v columns of qkv, exactly as inside rosa_generate_actions. */
rosa_status rosa_debug_attention(rosa_batch *b, const rosa_request *reqs, int32_t n, int32_t layer,
                                 const void *qkv, void *o);

/* One projection alone, on M stacked rows (M <= max_action_tokens).
 *   which = 0: out[M][Q]      = a[M][d] W_qkv[layer]                      (model dtype)
 *   which = 1: out[M][d]     += gate[M][d] * (a[M][n_q*hd] W_o[layer])     (fp32)
 *   which = 2: out[M][d_mlp]  = gelu_tanh(a[M][d] W_up[layer])             (model dtype)
 *   which = 3: out[M][d]     += gate[M][d] * (a[M][d_mlp] W_down[layer])   (fp32)
 * a is DEVICE in the model dtype; gate is DEVICE fp32 (ignored for 0 and 2).
 * a, out and gate must be 16-byte aligned (ROSA_E_INVALID otherwise). */
rosa_status rosa_debug_gemm(rosa_batch *b, int32_t which, int32_t layer, const void *a, int32_t M,
                            void *out, const float *gate);

/* Force the block configuration of every bf16 projection launched on this
 * handle (rosa_generate_actions and rosa_debug_gemm): cfg in [0, n) where n is
 * returned in *n_configs, or -1 for the built-in cost model (the default).
 * Every configuration computes each output with the same instruction sequence,
 * so results are bitwise identical whichever is used; only speed differs.
 * n_configs may be NULL. */
rosa_status rosa_debug_gemm_config(rosa_batch *b, int32_t cfg, int32_t *n_configs);

/* Number of lanes: a call with at least 64 requests per lane splits its
 * requests into that many sub-batches of similar work, each on its own stream
 * (the handle's stream for lane 0, internal default-priority streams for the
 * others), forked after the time conditioning and joined back on the handle's
 * stream before the call returns.  Requests are independent, so results are
 * bitwise identical for any lane count; only the overlap of the sub-batches'
 * kernels changes.  n in [1, 4]; the default is 2 in bf16 mode, 1 in fp32
 * mode.  While per-kernel profiling is enabled every call runs one lane. */
rosa_status rosa_debug_set_lanes(rosa_batch *b, int32_t n);

/* Per-kernel timing.  While enabled, every launch of the handle is bracketed
 * by HIP events on the handle's stream and its duration is added to its
 * kernel class.  rosa_debug_get_profile synchronizes the stream, then fills up
 * to max entries of names (static strings), launch counts and total
 * milliseconds, and sets *n_out.  Enabling clears the totals. */
rosa_status rosa_debug_set_profiling(rosa_batch *b, int32_t enable);
rosa_status rosa_debug_get_profile(rosa_batch *b, const char **names, int64_t *launches,
                                   double *total_ms, int32_t max, int32_t *n_out);

/* The same per-kernel timing for a prefix producer handle (rosa_prefill.h):
 * classes load, norm, gemm_qkv, kv_scatter, attention, attn_merge, gemm_o,
 * gemm_up, gemm_down. */
rosa_status rosa_debug_prefill_set_profiling(rosa_prefill *h, int32_t enable);
/* Force the prefix producer's projection block configuration (as
 * rosa_debug_gemm_config). */
rosa_status rosa_debug_prefill_gemm_config(rosa_prefill *h, int32_t cfg, int32_t *n_configs);
rosa_status rosa_debug_prefill_get_profile(rosa_prefill *h, const char **names, int64_t *launches,
                                           double *total_ms, int32_t max, int32_t *n_out);

#ifdef __cplusplus
}
#endif

#endif /* ROSA_DEBUG_H_ */
