"""CPU oracle for batched flow-matching action-chunk generation (test infrastructure).

This is the reference the GPU library is checked against.  It is deliberately
plain: NumPy float64 throughout, one request at a time, one Euler step at a
time, one layer at a time, with matrix products as the only library steps.
Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
it; the product path never calls it.

What is computed.  The paper (Sec. 2.2.1) describes System-1 action models as a
vision-language backbone whose cached prefix feeds an action-generation head
such as a diffusion transformer, and (Sec. 2.3) diffusion-style action experts
that run a small number of denoising steps.  Its serving system batches
System-1 requests from many robots into one call on a GPU worker (Sec. 3.2;
Sec. 3.4.1, batching decisions; Sec. 4.3, System-1 batching).  The paper does not write
out the action expert's layers, so the forward pass below follows these
readings (each is restated where it is used):

* flow matching integrated by explicit Euler from noise at tau = 0 to tau = 1:
  tau_k = k / K (fp32 division), dt = 1 / K, x <- x + dt * v(x, tau_k);
* sinusoidal time embedding [sin(1000 tau w_i) || cos(1000 tau w_i)],
  w_i = 10000^(-i/half), then Linear-SiLU-Linear, and SiLU of the result feeds
  every modulation projection;
* each block: adaLN-style modulation (shift, 1 + scale, gate) of an RMSNorm
  without learned gain (eps 1e-6), attention, gated residual, same for a plain
  two-matrix tanh-GELU MLP; no biases in QKV/O/MLP;
* attention: each action token of request r attends, bidirectionally, to all
  P_r cached prefix keys of request r followed by all H_r action keys of
  request r (the joint, pi0-style layout); scale 1/sqrt(head_dim); query head
  g reads KV head g // (n_q / n_kv); no rotary embedding.  The alternating,
  GR00T-style layout (a DiT head that interleaves cross-attention to the VLM
  context with self-attention, Sec. 2.2.1) attends to the prefix keys only in
  even layers and to the request's own action keys only in odd layers;
* final modulated RMSNorm (shift, scale) and an output projection with bias
  give the velocity.

Pins (tests marked ``not gpu``): brute-force scalar attention on tiny inputs;
single-key, equal-key and zero-query attention; the embedding at tau = 0 and
its sin^2 + cos^2 = 1 pairs; RMSNorm of a constant vector; tanh-GELU against
the erf GELU within the approximation's error bound; the Euler closed forms
(zero velocity, constant velocity); the zero-gate closed form of the whole
network; a scalar brute-force forward on a tiny model; batch and permutation
invariance.  Agreement with the paper's own models is unpinned: their weights
and outputs are not published.
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence

import numpy as np

F = np.float64


def tau_grid(num_steps: int) -> List[float]:
    """Flow time of each Euler step: tau_k = k / K, divided in fp32 (so that the
    GPU, which divides in fp32, sees the same value)."""
    return [float(np.float32(k) / np.float32(num_steps)) for k in range(num_steps)]


def timestep_embedding(tau: float, dim: int) -> np.ndarray:
    """Sinusoidal embedding of flow time: half = dim / 2 frequencies
    w_i = 10000^(-i / half); e = [sin(1000 tau w_i) for i] ++ [cos(1000 tau w_i) for i]."""
    half = dim // 2
    i = np.arange(half, dtype=F)
    w = np.power(F(10000.0), -i / F(half))
    arg = F(1000.0) * F(tau) * w
    return np.concatenate([np.sin(arg), np.cos(arg)])


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    """GELU, tanh approximation: 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x * x * x)))


def rms_norm(h: np.ndarray, eps: float) -> np.ndarray:
    """Row-wise RMSNorm without learned gain: h / sqrt(mean(h^2) + eps)."""
    ms = np.mean(h * h, axis=-1, keepdims=True)
    return h / np.sqrt(ms + eps)


def modulate(x: np.ndarray, shift: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """adaLN modulation: x * (1 + scale) + shift (shift/scale broadcast over rows)."""
    return x * (1.0 + scale) + shift


def softmax_rows(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Grouped-query attention of one request, no mask inside the request.

    q: [Tq][n_q][hd] queries; k, v: [Tk][n_kv][hd] keys/values (prefix keys
    first, then the action tokens' own keys).  Query head g uses KV head
    g // (n_q / n_kv).  Returns o: [Tq][n_q][hd]."""
    n_q, hd = q.shape[1], q.shape[2]
    n_kv = k.shape[1]
    group = n_q // n_kv
    o = np.empty_like(q)
    for g in range(n_q):
        j = g // group
        s = q[:, g, :] @ k[:, j, :].T / math.sqrt(hd)       # [Tq][Tk]
        o[:, g, :] = softmax_rows(s) @ v[:, j, :]
    return o


class OracleModel:
    """The action expert with its weights held in float64."""

    def __init__(self, weights: Dict[str, np.ndarray], shape):
        self.shape = shape
        self.w = {k: np.asarray(v, dtype=F) for k, v in weights.items()}

    # ---- time conditioning
    def time_condition(self, tau: float) -> np.ndarray:
        """s = SiLU(W_t2^T SiLU(W_t1^T e(tau) + b_t1) + b_t2): the vector every
        modulation projection reads."""
        w = self.w
        e = timestep_embedding(tau, self.shape.time_emb_dim)
        c = silu(e @ w["w_t1"] + w["b_t1"]) @ w["w_t2"] + w["b_t2"]
        return silu(c)

    def block_modulation(self, s: np.ndarray, layer: int):
        """(shift_attn, scale_attn, gate_attn, shift_mlp, scale_mlp, gate_mlp)."""
        m = s @ self.w["w_mod"][layer] + self.w["b_mod"][layer]
        return np.split(m, 6)

    def final_modulation(self, s: np.ndarray):
        """(shift, scale) of the final norm."""
        return np.split(s @ self.w["w_fmod"] + self.w["b_fmod"], 2)

    # ---- one velocity evaluation
    def attention_keys(self, l: int, prefix_k, prefix_v, ka: np.ndarray, va: np.ndarray):
        """Keys and values layer l's action tokens attend to.  Joint layout
        (pi0-style, 0): the request's prefix keys of layer l, then its own
        action keys.  Alternating layout (GR00T-style DiT, 1): even layers
        cross-attend to the prefix keys only, odd layers self-attend to the
        request's own action keys only."""
        pk = np.asarray(prefix_k[l], dtype=F) if len(prefix_k) else None
        pv = np.asarray(prefix_v[l], dtype=F) if len(prefix_v) else None
        if getattr(self.shape, "attention_layout", 0) == 1:
            return (pk, pv) if l % 2 == 0 else (ka, va)
        if pk is None or pk.shape[0] == 0:
            return ka, va
        return np.concatenate([pk, ka], axis=0), np.concatenate([pv, va], axis=0)

    def velocity(self, x: np.ndarray, tau: float, prefix_k: np.ndarray, prefix_v: np.ndarray
                 ) -> np.ndarray:
        """v(x, tau) for one request.  x: [H][A]; prefix_k/v: [L][P][n_kv][hd]."""
        sh, w = self.shape, self.w
        H = x.shape[0]
        nq, nkv, hd = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
        s = self.time_condition(tau)
        h = x @ w["w_in"] + w["b_in"]                               # [H][d]
        for l in range(sh.n_layers):
            sa, ca, ga, sm, cm, gm = self.block_modulation(s, l)
            u = modulate(rms_norm(h, sh.rms_eps), sa, ca)
            qkv = u @ w["w_qkv"][l]                                  # [H][(nq+2nkv)hd]
            q = qkv[:, : nq * hd].reshape(H, nq, hd)
            ka = qkv[:, nq * hd: (nq + nkv) * hd].reshape(H, nkv, hd)
            va = qkv[:, (nq + nkv) * hd:].reshape(H, nkv, hd)
            kf, vf = self.attention_keys(l, prefix_k, prefix_v, ka, va)
            o = attention(q, kf, vf).reshape(H, nq * hd)
            h = h + ga * (o @ w["w_o"][l])
            u = modulate(rms_norm(h, sh.rms_eps), sm, cm)
            h = h + gm * (gelu_tanh(u @ w["w_up"][l]) @ w["w_down"][l])
        sf, cf = self.final_modulation(s)
        return modulate(rms_norm(h, sh.rms_eps), sf, cf) @ w["w_out"] + w["b_out"]

    # ---- Euler integration of one request
    def generate_chunk(self, noise: np.ndarray, num_steps: int, prefix_k: np.ndarray,
                       prefix_v: np.ndarray) -> np.ndarray:
        """x_0 = noise; x_{k+1} = x_k + (1/K) v(x_k, k/K); returns x_K [H][A]."""
        x = np.asarray(noise, dtype=F).copy()
        dt = 1.0 / num_steps
        for tau in tau_grid(num_steps):
            x = x + dt * self.velocity(x, tau, prefix_k, prefix_v)
        return x

    def advance(self, x: np.ndarray, num_steps: int, k0: int, k1: int, prefix_k: np.ndarray,
                prefix_v: np.ndarray) -> np.ndarray:
        """Euler steps k0 .. k1-1 of the same grid from the state x_{k0}:
        returns x_{k1}.  Step-level batching (admission and retirement between
        steps, the continuous batching the paper applies to its
        autoregressive models, Sec. 3.4.1) only regroups these steps."""
        x = np.asarray(x, dtype=F).copy()
        dt = 1.0 / num_steps
        taus = tau_grid(num_steps)
        for k in range(k0, k1):
            x = x + dt * self.velocity(x, taus[k], prefix_k, prefix_v)
        return x

    def generate(self, requests: Sequence) -> List[np.ndarray]:
        """A batch is a list of independent requests; each result depends on its
        own request only."""
        out = []
        for r in requests:
            out.append(self.generate_chunk(r.noise, r.steps, r.prefix_f32("k"), r.prefix_f32("v")))
        return out
