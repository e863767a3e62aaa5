"""CPU oracle for the prefix producer (test infrastructure only).

The paper's System-1 models run a vision-language backbone over each robot's
observation and instruction, and its cached prefix feeds the action head
(Sec. 2.2.1: a VLM backbone followed by an action-generation head such as a
diffusion transformer).  The action expert reads, at layer l, the keys and
values the backbone's layer l produced for the prefix tokens.  The paper does
not write out the backbone; the reading taken here (each step restated where
it is used):

* input: the prefix tokens already embedded (image patches and text), [P][d];
* each layer: RMSNorm (eps 1e-6, no learned gain), fused QKV projection,
  optionally a rotary position embedding of the queries and keys (the
  shape's rope_base > 0: elements i and i + hd/2 of each head turn by the
  angle p base^(-2i/hd) at the token's index p within its job; the cache
  holds the turned keys), attention of every prefix token over the prefix
  tokens of its own request: all of them (bidirectional), or, when the job ends in a
  causal segment of c tokens, token t over tokens [0, max(P - c, t + 1)) (a
  prefix-LM mask: image patches and prompt see each other, the segment's
  tokens see those and the segment up to themselves), output projection and
  residual; RMSNorm, a plain two-matrix tanh-GELU MLP and residual; no biases;
* the layer's cache: its K and V projections of the prefix tokens,
  [L][P][n_kv][hd].

Plain NumPy float64, one request at a time, one layer at a time; matrix
products and the pinned attention, RMSNorm and GELU of ``rosa_oracle`` are
its only steps.

A second cache form serves an action head that cross-attends to the
backbone's output instead (a GR00T-style DiT head): ``prefill_context`` runs
every backbone layer, RMS-normalises the final hidden state and projects it
with each head layer's own context weights into that layer's K and V.

Pins (tests marked ``not gpu``): a scalar brute force on nested lists for a
tiny backbone (both cache forms, with and without a causal segment); with the
residual branches zeroed every layer's cache is the closed form RMSNorm(x)
W_k, W_v of that layer (context form: RMSNorm(x) W_ctx[e]); permuting the
prefix tokens permutes the cache rows (no causal segment, no positions).
Rotary embedding: the identity at position 0, a plain 2-D rotation by p
radians at head width 2, every (i, i + hd/2) pair's length kept, query-key
dot products that depend only on the positions' difference, and a scalar
brute force that turns each pair as a complex number.
With a causal segment: a token's caches do not change when the tokens it
cannot see are changed or dropped (the job cut after it, or, for the
bidirectional part, the segment removed), and a fully causal job's first
token has the caches of that token alone.
"""
from __future__ import annotations

from typing import Dict, Tuple

import numpy as np

from .rosa_oracle import attention, gelu_tanh, rms_norm, softmax_rows

F = np.float64


def rotary(x: np.ndarray, base: float) -> np.ndarray:
    """Rotary position embedding of x [P][heads][hd] at positions 0 .. P-1:
    in every head, elements i and i + hd/2 (i < hd/2) turn by the angle
    p * base^(-2 i / hd)."""
    P, _, hd = x.shape
    half = hd // 2
    freq = np.power(float(base), -2.0 * np.arange(half, dtype=F) / hd)
    ang = np.arange(P, dtype=F)[:, None] * freq[None, :]                 # [P][half]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def prefix_lm_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, causal_len: int) -> np.ndarray:
    """Grouped-query attention of one job's tokens over each other when its
    last causal_len tokens form a causal segment: token t sees tokens
    [0, max(P - causal_len, t + 1)).  causal_len = 0 is plain bidirectional
    attention."""
    if causal_len == 0:
        return attention(q, k, v)
    P, n_q, hd = q.shape
    n_kv = k.shape[1]
    group = n_q // n_kv
    b = P - causal_len
    t = np.arange(P)
    visible = t[None, :] < np.maximum(b, t + 1)[:, None]          # [query token][key token]
    o = np.empty_like(q)
    for g in range(n_q):
        j = g // group
        s = q[:, g, :] @ k[:, j, :].T / np.sqrt(hd)
        o[:, g, :] = softmax_rows(np.where(visible, s, -np.inf)) @ v[:, j, :]
    return o


def prefill(x: np.ndarray, w: Dict[str, np.ndarray], shape, causal_len: int = 0
            ) -> Tuple[np.ndarray, np.ndarray]:
    """Prefix caches (K, V), each [L][P][n_kv][hd] float64, of one request whose
    embedded prefix tokens are x [P][d] (the last causal_len of them a causal
    segment)."""
    L, nq, nkv, hd, eps = shape.n_layers, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.rms_eps
    rope = getattr(shape, "rope_base", 0.0)
    P = x.shape[0]
    h = np.asarray(x, dtype=F).copy()
    K = np.zeros((L, P, nkv, hd), dtype=F)
    V = np.zeros((L, P, nkv, hd), dtype=F)
    for l in range(L):
        qkv = rms_norm(h, eps) @ np.asarray(w["w_qkv"][l], dtype=F)
        q = qkv[:, :nq * hd].reshape(P, nq, hd)
        k = qkv[:, nq * hd:(nq + nkv) * hd].reshape(P, nkv, hd)
        v = qkv[:, (nq + nkv) * hd:].reshape(P, nkv, hd)
        if rope > 0:
            q, k = rotary(q, rope), rotary(k, rope)
        K[l], V[l] = k, v
        o = prefix_lm_attention(q, k, v, causal_len) if P > 0 else np.zeros((0, nq, hd), dtype=F)
        h = h + o.reshape(P, nq * hd) @ np.asarray(w["w_o"][l], dtype=F)
        u = rms_norm(h, eps)
        h = h + gelu_tanh(u @ np.asarray(w["w_up"][l], dtype=F)) @ np.asarray(w["w_down"][l], dtype=F)
    return K, V


def prefill_context(x: np.ndarray, w: Dict[str, np.ndarray], shape, w_ctx: np.ndarray, causal_len: int = 0
                    ) -> Tuple[np.ndarray, np.ndarray]:
    """Context caches (K, V), each [L_e][P][n_kv][hd] float64, for an action
    head that cross-attends to the backbone's output (the GR00T-style head):
    every backbone layer runs in full, the final hidden state is RMS-normalised
    (no gain), and action-head layer e projects it with its own context
    weights w_ctx[e] ([d][2 n_kv hd], K columns then V)."""
    L, nq, nkv, hd, eps = shape.n_layers, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.rms_eps
    rope = getattr(shape, "rope_base", 0.0)
    P = x.shape[0]
    h = np.asarray(x, dtype=F).copy()
    for l in range(L):
        qkv = rms_norm(h, eps) @ np.asarray(w["w_qkv"][l], dtype=F)
        q = qkv[:, :nq * hd].reshape(P, nq, hd)
        k = qkv[:, nq * hd:(nq + nkv) * hd].reshape(P, nkv, hd)
        v = qkv[:, (nq + nkv) * hd:].reshape(P, nkv, hd)
        if rope > 0:
            q, k = rotary(q, rope), rotary(k, rope)
        h = h + prefix_lm_attention(q, k, v, causal_len).reshape(P, nq * hd) @ np.asarray(w["w_o"][l], dtype=F)
        h = h + gelu_tanh(rms_norm(h, eps) @ np.asarray(w["w_up"][l], dtype=F)) @ np.asarray(w["w_down"][l], dtype=F)
    u = rms_norm(h, eps)
    Le = w_ctx.shape[0]
    K = np.zeros((Le, P, nkv, hd), dtype=F)
    V = np.zeros((Le, P, nkv, hd), dtype=F)
    for e in range(Le):
        kv = u @ np.asarray(w_ctx[e], dtype=F)
        K[e] = kv[:, :nkv * hd].reshape(P, nkv, hd)
        V[e] = kv[:, nkv * hd:].reshape(P, nkv, hd)
    return K, V
