/*
 * rosa_prefill.h - the prefix producer: a vision-language backbone over each
 * request's embedded prefix tokens, writing the per-layer keys and values
 * that rosa_generate_actions reads as the request's cached prefix.
 *
 * The paper's System-1 models are a VLM backbone whose cached prefix feeds an
 * action-generation head (Sec. 2.2.1); the action expert attends at layer l to
 * the keys and values the backbone's layer l produced for the prefix tokens.
 * The paper does not write out the backbone; the library takes this reading:
 *   h = the embedded prefix tokens (image patches and text, [P][d]);
 *   each layer l: u = RMSNorm(h) (eps = rms_eps, no learned gain);
 *     [q | k | v] = u W_qkv[l]; with rope_base > 0, q and k are rotated
 *       (rotary position embedding at the token's index p within its job:
 *       elements i and i + hd/2 of each head turn by p * rope_base^(-2i/hd));
 *     cache_k[l] = k, cache_v[l] = v;
 *     every prefix token attends to the prefix tokens of its own request
 *     (scale 1/sqrt(head_dim), query head g reads KV head
 *     g / (n_q / n_kv)): all of them (bidirectional), or, for a job with a
 *     causal segment of its last c tokens, token t sees tokens
 *     [0, max(P - c, t + 1)) (prefix-LM: the first P - c tokens, image patches
 *     and prompt, see each other; each later token sees those and the
 *     segment's tokens up to itself);  h += o W_o[l];
 *     h += gelu_tanh(RMSNorm(h) W_up[l]) W_down[l];
 *   no biases.
 * The backbone's n_layers, n_kv_heads and head_dim must equal the action
 * expert's for its caches to feed rosa_generate_actions.
 *
 * Same conventions as rosa.h: pure C, noexcept, status returns, asynchronous
 * on the handle's stream, all-or-nothing validation, a HIP failure poisons the
 * handle.  Precision as rosa_dtype: bf16 weights, embeddings, projections and
 * caches with fp32 accumulation and an fp32 residual stream (ROSA_BF16), or
 * everything fp32 (ROSA_FP32).
 */
#ifndef ROSA_PREFILL_H_
#define ROSA_PREFILL_H_

#include "rosa.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rosa_prefill rosa_prefill;   /* opaque handle */

/* What the caches hold.
 *  ROSA_CACHE_PER_LAYER: layer l's K and V projections of the prefix tokens
 *    (a pi0-style expert sharing the backbone's attention; the caches have
 *    n_layers layers).
 *  ROSA_CACHE_CONTEXT: context K and V for an action head that cross-attends
 *    to the backbone's output (GR00T-style, ROSA_ATTN_ALTERNATING): every
 *    backbone layer runs in full, the final hidden state is RMS-normalised
 *    (no gain), and head layer e projects it with w_ctx[e]; the caches have
 *    head_layers layers. */
typedef enum rosa_cache_form {
  ROSA_CACHE_PER_LAYER = 0,
  ROSA_CACHE_CONTEXT = 1
} rosa_cache_form;

/* Backbone shape.  Constraints (else ROSA_E_UNSUPPORTED): n_q_heads % n_kv_heads
 * == 0; head_dim in {32, 64, 128, 256}; d_model, d_mlp and n_q_heads*head_dim
 * multiples of 128; d_model <= 4096.  cache_form is a rosa_cache_form and
 * head_layers >= 1 with ROSA_CACHE_CONTEXT (ignored otherwise); else
 * ROSA_E_INVALID. */
typedef struct rosa_vlm_config {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t d_mlp;
  float   rms_eps;
  int32_t dtype;           /* rosa_dtype */
  int32_t cache_form;      /* rosa_cache_form */
  int32_t head_layers;     /* ROSA_CACHE_CONTEXT: layers of the action head (L_e) */
  float   rope_base;       /* > 1: rotary position embedding of the backbone's
                              queries and keys with this base (10000 in Gemma);
                              0: no positions; else ROSA_E_INVALID */
} rosa_vlm_config;

/* Weights: HOST float32, row-major [in][out] (y = x W), L = n_layers, d = d_model,
 * Q = (n_q + 2 n_kv) head_dim, q columns first, then k, then v.  Copied and
 * repacked by create; the caller may free them afterwards. */
typedef struct rosa_vlm_weights {
  const float *w_qkv;      /* [L][d][Q] */
  const float *w_o;        /* [L][n_q head_dim][d] */
  const float *w_up;       /* [L][d][d_mlp] */
  const float *w_down;     /* [L][d_mlp][d] */
  const float *w_ctx;      /* ROSA_CACHE_CONTEXT: [L_e][d][2 n_kv head_dim], K columns
                              then V; ignored (may be NULL) otherwise */
} rosa_vlm_weights;

/* One request's prefix.  DEVICE pointers owned by the caller, valid until the
 * stream has passed the call.
 *   embeddings: [P][d] in the model dtype (read only);
 *   prefix_k, prefix_v: [L_c][P][n_kv][head_dim] in the model dtype, written
 *       (the layout rosa_request.prefix_k / prefix_v expects); L_c = n_layers
 *       (ROSA_CACHE_PER_LAYER) or head_layers (ROSA_CACHE_CONTEXT).      */
typedef struct rosa_prefix_job {
  const void *embeddings;
  void       *prefix_k;
  void       *prefix_v;
  int32_t     prefix_len;  /* P >= 1 */
  int32_t     causal_len;  /* c, 0 <= c <= P: the last c tokens form a causal
                              segment (see the layer above); 0 = all
                              bidirectional */
} rosa_prefix_job;

/* Create a handle: validate, upload and repack the weights, allocate
 * workspaces for up to max_jobs jobs and max_tokens prefix tokens per call.
 * hip_stream: a hipStream_t (NULL = the default stream).  Errors as
 * rosa_batch_create; *out is NULL on failure. */
rosa_status rosa_prefill_create(const rosa_vlm_config *cfg, const rosa_vlm_weights *w, int32_t max_jobs,
                                int64_t max_tokens, void *hip_stream, rosa_prefill **out);

/* Run the backbone over n jobs (a ragged batch: each job's tokens attend only
 * to their own prefix) and write every layer's caches.  n == 0 is a no-op.
 * Errors: ROSA_E_INVALID (NULL pointers, P < 1, causal_len outside [0, P]),
 * ROSA_E_CAPACITY (n or the sum of P above the capacity), ROSA_E_DEVICE. */
rosa_status rosa_prefill_run(rosa_prefill *h, const rosa_prefix_job *jobs, int32_t n);

/* Wait for the handle's stream, then free everything.  NULL-safe. */
void rosa_prefill_destroy(rosa_prefill *h);

/* Detail of the last failure on this handle ("" if none); with h == NULL the
 * last failure of a create. */
const char *rosa_prefill_last_error(const rosa_prefill *h);

#ifdef __cplusplus
}
#endif

#endif /* ROSA_PREFILL_H_ */
