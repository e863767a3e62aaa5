"""Pins of the prefix-producer oracle (Sec. 2.2.1: the VLM backbone's per-layer
keys and values are the action head's prefix cache).  No GPU needed."""
import cmath
import dataclasses
import math

import numpy as np

from oracle import prefill, prefill_context
from oracle.prefill import rotary
from synthetic import TINY_VLM, VlmShape, make_context_weights, make_prefix_embeddings, make_vlm_weights

SMALL = VlmShape(n_layers=2, d_model=8, n_q_heads=4, n_kv_heads=2, head_dim=4, d_mlp=12)


def _brute_prefill(x, w, s, causal_len=0):
    """Scalar brute force on nested Python lists.  With a causal segment of the
    last causal_len tokens, key u is visible to token t when u lies before the
    segment or u <= t.  With s.rope_base > 0 each (i, i + hd/2) pair of a query
    or key head at position t is the complex number x_i + j x_(i+hd/2) times
    exp(j t rope_base^(-2i/hd))."""
    L, d, nq, nkv, hd, dff = s.n_layers, s.d_model, s.n_q_heads, s.n_kv_heads, s.head_dim, s.d_mlp
    G = nq // nkv
    P = len(x)
    h = [[float(v) for v in row] for row in x]

    def norm(row):
        ms = sum(v * v for v in row) / len(row)
        return [v / math.sqrt(ms + s.rms_eps) for v in row]

    def matvec(row, W):
        return [sum(row[i] * float(W[i][j]) for i in range(len(row))) for j in range(len(W[0]))]

    Ks, Vs = [], []
    for l in range(L):
        qkv = [matvec(norm(row), w["w_qkv"][l]) for row in h]
        q = [[r[g * hd:(g + 1) * hd] for g in range(nq)] for r in qkv]
        k = [[r[(nq + j) * hd:(nq + j + 1) * hd] for j in range(nkv)] for r in qkv]
        if s.rope_base > 0:
            def turn(vec, t):
                half = hd // 2
                out = [0.0] * hd
                for i in range(half):
                    z = complex(vec[i], vec[i + half]) * cmath.exp(1j * t * s.rope_base ** (-2.0 * i / hd))
                    out[i], out[i + half] = z.real, z.imag
                return out
            q = [[turn(head, t) for head in q[t]] for t in range(P)]
            k = [[turn(head, t) for head in k[t]] for t in range(P)]
        v = [[r[(nq + nkv + j) * hd:(nq + nkv + j + 1) * hd] for j in range(nkv)] for r in qkv]
        Ks.append(k)
        Vs.append(v)
        o = []
        for t in range(P):
            row = []
            for g in range(nq):
                j = g // G
                keys = [u for u in range(P) if u < P - causal_len or u <= t]
                sc = [sum(q[t][g][e] * k[u][j][e] for e in range(hd)) / math.sqrt(hd) for u in keys]
                m = max(sc)
                ex = [math.exp(z - m) for z in sc]
                tot = sum(ex)
                row += [sum(ex[i] * v[u][j][e] for i, u in enumerate(keys)) / tot for e in range(hd)]
            o.append(row)
        h = [[a + b for a, b in zip(hr, matvec(orow, w["w_o"][l]))] for hr, orow in zip(h, o)]
        new = []
        for hr in h:
            up = matvec(norm(hr), w["w_up"][l])
            gl = [0.5 * z * (1.0 + math.tanh(math.sqrt(2.0 / math.pi) * (z + 0.044715 * z ** 3))) for z in up]
            new.append([a + b for a, b in zip(hr, matvec(gl, w["w_down"][l]))])
        h = new
    return np.array(Ks), np.array(Vs), h


def test_prefill_matches_scalar_bruteforce():
    rng = np.random.default_rng(0)
    w = {k: rng.standard_normal(v.shape) * 0.5 for k, v in make_vlm_weights(SMALL, "fp32").items()}
    x = rng.standard_normal((5, SMALL.d_model))
    K, V = prefill(x, w, SMALL)
    Kb, Vb, _ = _brute_prefill(x, w, SMALL)
    np.testing.assert_allclose(K, Kb, rtol=0, atol=1e-11)
    np.testing.assert_allclose(V, Vb, rtol=0, atol=1e-11)


def test_zero_residual_branches_give_per_layer_closed_form():
    w = make_vlm_weights(TINY_VLM, "fp32", seed=4)
    w["w_o"][:] = 0.0
    w["w_down"][:] = 0.0
    x = make_prefix_embeddings(TINY_VLM, 9, "fp32", seed=5).astype(np.float64)
    K, V = prefill(x, w, TINY_VLM)
    nq, nkv, hd = TINY_VLM.n_q_heads, TINY_VLM.n_kv_heads, TINY_VLM.head_dim
    u = x / np.sqrt((x * x).mean(axis=1, keepdims=True) + TINY_VLM.rms_eps)
    for l in range(TINY_VLM.n_layers):
        qkv = u @ w["w_qkv"][l].astype(np.float64)
        np.testing.assert_allclose(K[l], qkv[:, nq * hd:(nq + nkv) * hd].reshape(9, nkv, hd), rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(V[l], qkv[:, (nq + nkv) * hd:].reshape(9, nkv, hd), rtol=1e-12, atol=1e-13)


def test_token_permutation_permutes_the_cache():
    w = make_vlm_weights(TINY_VLM, "fp32", seed=6)
    x = make_prefix_embeddings(TINY_VLM, 12, "fp32", seed=7).astype(np.float64)
    perm = np.random.default_rng(8).permutation(12)
    K, V = prefill(x, w, TINY_VLM)
    Kp, Vp = prefill(x[perm], w, TINY_VLM)
    np.testing.assert_allclose(Kp, K[:, perm], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(Vp, V[:, perm], rtol=1e-12, atol=1e-13)


def test_context_form_matches_scalar_bruteforce():
    rng = np.random.default_rng(1)
    w = {k: rng.standard_normal(v.shape) * 0.5 for k, v in make_vlm_weights(SMALL, "fp32").items()}
    wc = rng.standard_normal((3, SMALL.d_model, 2 * SMALL.n_kv_heads * SMALL.head_dim)) * 0.5
    x = rng.standard_normal((4, SMALL.d_model))
    K, V = prefill_context(x, w, SMALL, wc)
    _, _, h = _brute_prefill(x, w, SMALL)
    kvw = SMALL.n_kv_heads * SMALL.head_dim
    for e in range(3):
        for t in range(4):
            ms = sum(z * z for z in h[t]) / len(h[t])
            u = [z / math.sqrt(ms + SMALL.rms_eps) for z in h[t]]
            kv = [sum(u[i] * wc[e][i][j] for i in range(len(u))) for j in range(2 * kvw)]
            np.testing.assert_allclose(K[e, t].reshape(-1), kv[:kvw], rtol=0, atol=1e-11)
            np.testing.assert_allclose(V[e, t].reshape(-1), kv[kvw:], rtol=0, atol=1e-11)


def test_context_form_zero_residual_closed_form_and_permutation():
    w = make_vlm_weights(TINY_VLM, "fp32", seed=4)
    wc = make_context_weights(TINY_VLM, 3, "fp32")
    x = make_prefix_embeddings(TINY_VLM, 9, "fp32", seed=5).astype(np.float64)
    z = {k: v.copy() for k, v in w.items()}
    z["w_o"][:] = 0.0
    z["w_down"][:] = 0.0
    K, V = prefill_context(x, z, TINY_VLM, wc)
    kvw = TINY_VLM.n_kv_heads * TINY_VLM.head_dim
    u = x / np.sqrt((x * x).mean(axis=1, keepdims=True) + TINY_VLM.rms_eps)
    for e in range(3):
        kv = u @ wc[e].astype(np.float64)
        np.testing.assert_allclose(K[e].reshape(9, kvw), kv[:, :kvw], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(V[e].reshape(9, kvw), kv[:, kvw:], rtol=1e-12, atol=1e-13)
    perm = np.random.default_rng(9).permutation(9)
    K1, V1 = prefill_context(x, w, TINY_VLM, wc)
    Kp, Vp = prefill_context(x[perm], w, TINY_VLM, wc)
    np.testing.assert_allclose(Kp, K1[:, perm], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(Vp, V1[:, perm], rtol=1e-12, atol=1e-13)


def test_causal_segment_matches_scalar_bruteforce():
    rng = np.random.default_rng(2)
    w = {k: rng.standard_normal(v.shape) * 0.5 for k, v in make_vlm_weights(SMALL, "fp32").items()}
    x = rng.standard_normal((5, SMALL.d_model))
    for c in (1, 3, 5):
        K, V = prefill(x, w, SMALL, causal_len=c)
        Kb, Vb, _ = _brute_prefill(x, w, SMALL, causal_len=c)
        np.testing.assert_allclose(K, Kb, rtol=0, atol=1e-11)
        np.testing.assert_allclose(V, Vb, rtol=0, atol=1e-11)


def test_causal_caches_ignore_the_tokens_they_cannot_see():
    # P = 12 with a causal segment of 5: tokens 0..6 see each other only, token
    # t >= 7 sees tokens 0..t.  Cutting the job after token t (t >= 7) keeps
    # tokens 0..t's caches; dropping the segment keeps tokens 0..6's; changing
    # the last token changes no other token's caches.
    w = make_vlm_weights(TINY_VLM, "fp32", seed=11)
    x = make_prefix_embeddings(TINY_VLM, 12, "fp32", seed=12).astype(np.float64)
    K, V = prefill(x, w, TINY_VLM, causal_len=5)
    for t in range(7, 12):
        Kt, Vt = prefill(x[:t + 1], w, TINY_VLM, causal_len=t + 1 - 7)
        np.testing.assert_allclose(Kt, K[:, :t + 1], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(Vt, V[:, :t + 1], rtol=1e-12, atol=1e-13)
    Kb, Vb = prefill(x[:7], w, TINY_VLM)
    np.testing.assert_allclose(Kb, K[:, :7], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(Vb, V[:, :7], rtol=1e-12, atol=1e-13)
    x2 = x.copy()
    x2[11] = -x2[11]
    K2, V2 = prefill(x2, w, TINY_VLM, causal_len=5)
    np.testing.assert_allclose(K2[:, :11], K[:, :11], rtol=1e-12, atol=1e-13)
    assert np.abs(K2[1:, 11] - K[1:, 11]).max() > 1e-3     # the changed token itself does change
    # Without the segment every token sees the last one.
    Kf, _ = prefill(x, w, TINY_VLM)
    Kf2, _ = prefill(x2, w, TINY_VLM)
    assert np.abs(Kf2[1:, 0] - Kf[1:, 0]).max() > 1e-6


def test_fully_causal_first_token_is_alone():
    w = make_vlm_weights(TINY_VLM, "fp32", seed=13)
    x = make_prefix_embeddings(TINY_VLM, 6, "fp32", seed=14).astype(np.float64)
    K, V = prefill(x, w, TINY_VLM, causal_len=6)
    K1, V1 = prefill(x[:1], w, TINY_VLM)
    np.testing.assert_allclose(K[:, :1], K1, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(V[:, :1], V1, rtol=1e-12, atol=1e-13)


def test_context_form_causal_matches_scalar_bruteforce():
    rng = np.random.default_rng(3)
    w = {k: rng.standard_normal(v.shape) * 0.5 for k, v in make_vlm_weights(SMALL, "fp32").items()}
    wc = rng.standard_normal((2, SMALL.d_model, 2 * SMALL.n_kv_heads * SMALL.head_dim)) * 0.5
    x = rng.standard_normal((5, SMALL.d_model))
    K, V = prefill_context(x, w, SMALL, wc, causal_len=2)
    _, _, h = _brute_prefill(x, w, SMALL, causal_len=2)
    kvw = SMALL.n_kv_heads * SMALL.head_dim
    for e in range(2):
        for t in range(5):
            ms = sum(z * z for z in h[t]) / len(h[t])
            u = [z / math.sqrt(ms + SMALL.rms_eps) for z in h[t]]
            kv = [sum(u[i] * wc[e][i][j] for i in range(len(u))) for j in range(2 * kvw)]
            np.testing.assert_allclose(K[e, t].reshape(-1), kv[:kvw], rtol=0, atol=1e-11)
            np.testing.assert_allclose(V[e, t].reshape(-1), kv[kvw:], rtol=0, atol=1e-11)


SMALL_ROPE = dataclasses.replace(SMALL, rope_base=10000.0)


def test_rotary_identity_at_zero_and_plain_rotation_at_width_two():
    rng = np.random.default_rng(20)
    x = rng.standard_normal((7, 3, 8))
    y = rotary(x, 10000.0)
    np.testing.assert_array_equal(y[0], x[0])                       # position 0: angle 0
    # head width 2: the single pair turns by p radians (base^0 = 1)
    x2 = rng.standard_normal((9, 1, 2))
    y2 = rotary(x2, 500.0)
    for p in range(9):
        c, s = math.cos(p), math.sin(p)
        a, b = x2[p, 0]
        np.testing.assert_allclose(y2[p, 0], [a * c - b * s, b * c + a * s], rtol=0, atol=1e-14)


def test_rotary_keeps_pair_lengths_and_depends_on_relative_position():
    rng = np.random.default_rng(21)
    hd, P = 16, 40
    x = rng.standard_normal((P, 2, hd))
    y = rotary(x, 10000.0)
    half = hd // 2
    np.testing.assert_allclose(np.hypot(y[..., :half], y[..., half:]), np.hypot(x[..., :half], x[..., half:]),
                               rtol=1e-13)
    # the same query and key vectors at every position: q_m . k_n depends on m - n only
    qv, kv = rng.standard_normal(hd), rng.standard_normal(hd)
    rq = rotary(np.tile(qv, (P, 1, 1)), 10000.0)[:, 0]
    rk = rotary(np.tile(kv, (P, 1, 1)), 10000.0)[:, 0]
    dots = rq @ rk.T
    for d in (-5, 0, 3, 17):
        diag = np.array([dots[m, m - d] for m in range(max(0, d), min(P, P + d))])
        np.testing.assert_allclose(diag, diag[0], rtol=1e-11, atol=1e-11)
    assert abs(dots[5, 2] - dots[5, 3]) > 1e-6                      # and it does depend on it


def test_rotary_prefill_matches_scalar_bruteforce():
    rng = np.random.default_rng(22)
    w = {k: rng.standard_normal(v.shape) * 0.5 for k, v in make_vlm_weights(SMALL_ROPE, "fp32").items()}
    x = rng.standard_normal((6, SMALL_ROPE.d_model))
    for c in (0, 2):
        K, V = prefill(x, w, SMALL_ROPE, causal_len=c)
        Kb, Vb, _ = _brute_prefill(x, w, SMALL_ROPE, causal_len=c)
        np.testing.assert_allclose(K, Kb, rtol=0, atol=1e-11)
        np.testing.assert_allclose(V, Vb, rtol=0, atol=1e-11)
    # positions take effect: permuting the tokens no longer permutes the cache
    perm = np.array([1, 0, 2, 3, 4, 5])
    Kp, _ = prefill(x[perm], w, SMALL_ROPE)
    K0, _ = prefill(x, w, SMALL_ROPE)
    assert np.abs(Kp[:, perm] - K0).max() > 1e-6


def test_rotary_context_form_matches_scalar_bruteforce():
    rng = np.random.default_rng(23)
    w = {k: rng.standard_normal(v.shape) * 0.5 for k, v in make_vlm_weights(SMALL_ROPE, "fp32").items()}
    wc = rng.standard_normal((2, SMALL_ROPE.d_model, 2 * SMALL_ROPE.n_kv_heads * SMALL_ROPE.head_dim)) * 0.5
    x = rng.standard_normal((5, SMALL_ROPE.d_model))
    K, V = prefill_context(x, w, SMALL_ROPE, wc)
    _, _, h = _brute_prefill(x, w, SMALL_ROPE)
    kvw = SMALL_ROPE.n_kv_heads * SMALL_ROPE.head_dim
    for e in range(2):
        for t in range(5):
            ms = sum(z * z for z in h[t]) / len(h[t])
            u = [z / math.sqrt(ms + SMALL_ROPE.rms_eps) for z in h[t]]
            kv = [sum(u[i] * wc[e][i][j] for i in range(len(u))) for j in range(2 * kvw)]
            np.testing.assert_allclose(K[e, t].reshape(-1), kv[:kvw], rtol=0, atol=1e-11)
            np.testing.assert_allclose(V[e, t].reshape(-1), kv[kvw:], rtol=0, atol=1e-11)
