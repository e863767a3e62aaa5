/*
 * rosa.h - batched flow-matching action-chunk generation on one AMD MI355X (gfx950).
 *
 * One call serves a batch of robot requests with a shared action expert, the
 * System-1 model of the paper's serving system: many robots' action-model
 * requests are batched into one call on one GPU worker (Sec. 3.2, inter-robot
 * batching on a shared pool; Sec. 3.4.1, batching decisions; Sec. 4.3, System-1
 * batching).
 * Each request brings its own cached vision-language prefix (keys and values
 * of every layer), an initial noise action chunk and a number of denoising
 * steps (Sec. 2.2.1: a VLM backbone feeds a diffusion-transformer action head;
 * Sec. 2.3: diffusion action experts run a few denoising steps), and gets back
 * its action chunk.
 *
 * The action expert computes, for every request independently:
 *   x_0 = noise;  x_{k+1} = x_k + (1/K) v(x_k, k/K),  k = 0..K-1;  result x_K
 * where v is a transformer over the request's H action tokens: sinusoidal
 * time embedding -> Linear/SiLU/Linear -> SiLU -> per-block modulation
 * (shift, scale, gate for attention and MLP); each block applies RMSNorm
 * (eps = rms_eps, no learned gain) modulated as norm*(1+scale)+shift,
 * grouped-query attention of the action tokens over [own prefix keys ; own
 * action keys] (or, in the alternating layout, over the prefix keys in even
 * layers and the action keys in odd layers) with scale 1/sqrt(head_dim), a
 * gated residual, then the same
 * around a tanh-GELU MLP; a final modulated RMSNorm and an output projection
 * with bias give v.  The paper does not spell out these layers; the library
 * follows the readings above, which its CPU oracle states one by one.
 *
 * Conventions
 *  - Pure C ABI.  No C++ or HIP types cross it; a HIP stream is passed as void*.
 *  - Every function is noexcept and returns a status (or nothing for destroy).
 *  - Validation is all-or-nothing: an invalid argument returns before any work
 *    is enqueued.  A HIP failure returns ROSA_E_DEVICE and poisons the handle;
 *    afterwards every call on it returns ROSA_E_DEVICE and only rosa_destroy
 *    is meaningful.
 *  - rosa_generate_actions is asynchronous on the handle's stream; outputs are
 *    valid once that stream has passed the call.  A handle is not thread-safe.
 */
#ifndef ROSA_H_
#define ROSA_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rosa_batch rosa_batch;   /* opaque handle */

typedef enum rosa_status {
  ROSA_OK = 0,
  ROSA_E_INVALID = 1,      /* bad argument (NULL pointer, bad size, bad count) */
  ROSA_E_CAPACITY = 2,     /* request set exceeds the capacity given at create */
  ROSA_E_NOMEM = 3,        /* device or pinned-host allocation failed */
  ROSA_E_DEVICE = 4,       /* HIP runtime failure, or the handle is poisoned */
  ROSA_E_UNSUPPORTED = 5   /* a shape the kernels do not implement */
} rosa_status;

typedef enum rosa_dtype {
  ROSA_BF16 = 0,   /* bf16 weights, prefix KV and activations; fp32 accumulation,
                      fp32 softmax statistics, fp32 residual stream and Euler state */
  ROSA_FP32 = 1    /* everything fp32 (debug mode, for tight parity checks) */
} rosa_dtype;

/* Attention layout of the action expert's blocks.
 *  ROSA_ATTN_JOINT: every layer attends over [own prefix keys ; own action
 *    keys] (a pi0-style expert sharing the VLM's attention).
 *  ROSA_ATTN_ALTERNATING: a DiT head that interleaves cross-attention to the
 *    VLM context with self-attention (GR00T-style, Sec. 2.2.1): even layers
 *    attend over the request's prefix keys only, odd layers over its own
 *    action keys only.  Every request needs prefix_len >= 1; the prefix cache
 *    keeps the [L][P][n_kv][hd] layout and odd layers' entries are not read. */
typedef enum rosa_attention_layout {
  ROSA_ATTN_JOINT = 0,
  ROSA_ATTN_ALTERNATING = 1
} rosa_attention_layout;

/* Model shape.  Constraints (else ROSA_E_UNSUPPORTED): n_q_heads % n_kv_heads == 0;
 * head_dim in {32, 64, 128, 256}; d_model, d_mlp and n_q_heads*head_dim multiples
 * of 128; d_model <= 4096; 1 <= action_dim <= 64; time_emb_dim even and <= 8192.
 * attention_layout is a rosa_attention_layout (else ROSA_E_INVALID). */
typedef struct rosa_model_config {
  int32_t n_layers;
  int32_t d_model;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t d_mlp;
  int32_t action_dim;
  int32_t time_emb_dim;
  float   rms_eps;
  int32_t dtype;           /* rosa_dtype */
  int32_t attention_layout;  /* rosa_attention_layout */
} rosa_model_config;

/* Weights: HOST float32 arrays, row-major [in][out] (y = x W), L = n_layers,
 * d = d_model, A = action_dim, dt = time_emb_dim, Q = (n_q + 2 n_kv) head_dim.
 * rosa_batch_create copies, converts (to bf16 in ROSA_BF16 mode, round to
 * nearest even) and repacks them; the caller may free them on return.
 * The fused QKV columns are [q heads 0..n_q-1 | k heads | v heads], each head
 * head_dim wide.  The modulation columns of layer l are
 * [shift_attn | scale_attn | gate_attn | shift_mlp | scale_mlp | gate_mlp],
 * each d wide; the final modulation is [shift | scale].                       */
typedef struct rosa_weights {
  const float *w_in, *b_in;        /* [A][d], [d]               input projection  */
  const float *w_t1, *b_t1;        /* [dt][d], [d]              time MLP layer 1  */
  const float *w_t2, *b_t2;        /* [d][d], [d]               time MLP layer 2  */
  const float *w_mod, *b_mod;      /* [L][d][6d], [L][6d]       block modulation  */
  const float *w_qkv;              /* [L][d][Q]                 fused QKV (no bias) */
  const float *w_o;                /* [L][n_q*head_dim][d]      attention output  */
  const float *w_up;               /* [L][d][d_mlp]             MLP up (no bias)  */
  const float *w_down;             /* [L][d_mlp][d]             MLP down (no bias) */
  const float *w_fmod, *b_fmod;    /* [d][2d], [2d]             final modulation  */
  const float *w_out, *b_out;      /* [d][A], [A]               velocity head     */
} rosa_weights;

/* Limits fixed at create; workspaces are sized from them. */
typedef struct rosa_capacity {
  int32_t max_requests;        /* requests per call */
  int32_t max_horizon;         /* H of any request */
  int32_t max_action_tokens;   /* sum of H over a call */
  int32_t max_steps;           /* K of any request (<= 64) */
  int64_t max_prefix_tokens;   /* sum of P over a call */
} rosa_capacity;

/* One robot request.  All pointers are DEVICE pointers owned by the caller and
 * must stay valid until the stream has passed the call.
 *   prefix_k, prefix_v: the request's cached prefix, layout [L][P][n_kv][head_dim]
 *       in the model dtype (bf16 or fp32), contiguous; layer stride P*n_kv*head_dim.
 *       Read only.  May be NULL when P == 0.  Several requests may share them.
 *   noise:   [H][A] fp32, the initial action chunk x_0 (read when start_step
 *            is 0; may be NULL otherwise).
 *   actions: [H][A] fp32, receives the Euler state after the last step the call
 *            runs for this request: x_K once every step is done.  When
 *            start_step > 0 it must hold x_{start_step}, as a previous call left
 *            it.  May alias noise.
 *   start_step: Euler steps already done (0 <= start_step < K): a request can
 *            be advanced over several calls and join a batch between steps.   */
typedef struct rosa_request {
  const void  *prefix_k;
  const void  *prefix_v;
  const float *noise;
  float       *actions;
  int32_t      prefix_len;    /* P >= 0 (>= 1 with ROSA_ATTN_ALTERNATING) */
  int32_t      horizon;       /* 1 <= H <= max_horizon */
  int32_t      num_steps;     /* 1 <= K <= max_steps; dt = 1/K, tau_k = k/K */
  int32_t      start_step;    /* 0 <= start_step < K */
} rosa_request;

/* Create a handle: validate the configuration, upload and repack the weights,
 * allocate workspaces for `cap`.  hip_stream is a hipStream_t (NULL = the
 * default stream); all work of this handle is enqueued on it.
 * Returns ROSA_E_INVALID for NULL arguments or non-positive sizes,
 * ROSA_E_UNSUPPORTED for shapes outside the constraints above, ROSA_E_NOMEM or
 * ROSA_E_DEVICE for allocation or HIP failures.  *out is NULL on failure. */
rosa_status rosa_batch_create(const rosa_model_config *cfg, const rosa_weights *w,
                              const rosa_capacity *cap, void *hip_stream, rosa_batch **out);

/* Generate the action chunks of n_reqs requests (the batch), asynchronously on
 * the handle's stream: every request runs its Euler steps start_step .. K-1.
 * Requests may differ in P, H, K and start_step; each result equals that
 * request computed alone (up to floating-point summation order).
 * n_reqs == 0 is a no-op returning ROSA_OK.  Errors: ROSA_E_INVALID (NULL
 * pointers, P < 0, H < 1, K < 1, H > max_horizon, K > max_steps, start_step
 * outside [0, K), NULL prefix with P > 0, NULL noise with start_step 0),
 * ROSA_E_CAPACITY (n_reqs, sum H or sum P above the capacity), ROSA_E_DEVICE
 * (HIP failure or poisoned handle). */
rosa_status rosa_generate_actions(rosa_batch *b, const rosa_request *reqs, int32_t n_reqs);

/* Step-level batching: like rosa_generate_actions, but each request runs at
 * most max_steps (>= 1) of its remaining steps, from start_step, and its
 * actions buffer receives the state after the last of them.  A caller that
 * advances a set of requests a step or a few at a time can admit new requests
 * (start_step 0) and retire finished ones (start_step + steps run == K)
 * between calls, so a request never waits for a whole batch to finish.  The
 * paper batches its autoregressive models this way (continuous batching) and
 * System-1 in discrete batches (Sec. 3.4.1); for the flow-matching expert the
 * Euler steps are the natural boundaries.  Errors as rosa_generate_actions,
 * and ROSA_E_INVALID for max_steps < 1. */
rosa_status rosa_generate_steps(rosa_batch *b, const rosa_request *reqs, int32_t n_reqs, int32_t max_steps);

/* Wait for the handle's stream, then free everything.  NULL-safe. */
void rosa_destroy(rosa_batch *b);

/* Ragged prefix + action attention of one layer that allocates nothing: for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).  It needs no handle.
 * Computes exactly what rosa_generate_actions computes at layer `layer` of
 * cfg's expert: each action token of request r attends over r's prefix keys
 * and values of that layer followed by r's own action keys and values (or,
 * with ROSA_ATTN_ALTERNATING, the prefix in even layers and the action keys in
 * odd layers), grouped-query heads, scale 1/sqrt(head_dim).
 *   reqs[n]: prefix_k / prefix_v / prefix_len / horizon / num_steps are read
 *            and validated as in rosa_generate_actions (noise and actions are
 *            not touched); rows follow the caller's request order.
 *   qkv: DEVICE [sum H][(n_q+2n_kv)*head_dim] in cfg's dtype, 16-byte aligned:
 *        the fused q | k | v projection of every request's action tokens.
 *   o:   DEVICE [sum H][n_q*head_dim] in cfg's dtype, 16-byte aligned, written.
 *   hip_stream: hipStream_t the work is enqueued on (NULL = default stream).
 * The plan of the call and the partial results of key ranges split over
 * several work items live in a library-owned device array of 16.7 MiB per GPU
 * (obtained once per device, held until the process ends): at most 1024
 * requests, 4096 attention work items and 64 split partials per call (fewer
 * key splits are made than rosa_generate_actions would make for a small
 * batch, so results can differ from it by rounding).  Every call on one GPU
 * reuses that array, so calls that overlap on a GPU (other streams, other
 * host threads) race; stream-ordered calls do not.  The plan is copied from
 * host memory with hipMemcpyAsync.  Errors: ROSA_E_INVALID, ROSA_E_UNSUPPORTED
 * (as rosa_batch_create for cfg, as rosa_generate_actions for the requests;
 * also misaligned qkv / o or a layer outside [0, n_layers)), ROSA_E_CAPACITY
 * (beyond the limits above), ROSA_E_DEVICE (HIP failure); rosa_last_error(NULL)
 * gives the detail.  n == 0 is a no-op. */
rosa_status rosa_attention_noalloc(const rosa_model_config *cfg, const rosa_request *reqs, int32_t n,
                                   int32_t layer, const void *qkv, void *o, void *hip_stream);

/* Static text for a status code. */
const char *rosa_status_string(rosa_status s);

/* Detail of the last failure on this handle ("" if none); valid until the
 * next call on the handle.  With b == NULL: the last failure of a create. */
const char *rosa_last_error(const rosa_batch *b);

#ifdef __cplusplus
}
#endif

#endif /* ROSA_H_ */
