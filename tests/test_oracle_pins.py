"""Pins for the CPU oracle against facts that do not come from the oracle itself:
brute force on tiny inputs, closed forms, special cases and invariants."""
import dataclasses
import math

import numpy as np
import pytest

from oracle import (OracleModel, attention, gelu_tanh, rms_norm, silu, tau_grid, timestep_embedding)
from synthetic import ModelShape, TINY_SHAPE, custom_request, make_weights

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")

MICRO = ModelShape(n_layers=2, d_model=8, n_q_heads=2, n_kv_heads=1, head_dim=4, d_mlp=16,
                   action_dim=3, time_emb_dim=6)


# ------------------------------------------------------------------ attention

def _attention_scalar(q, k, v):
    """Attention written out with scalar loops and math.exp (float64)."""
    Tq, nq, hd = q.shape
    Tk, nkv, _ = k.shape
    grp = nq // nkv
    out = np.zeros_like(q)
    for t in range(Tq):
        for g in range(nq):
            j = g // grp
            logits = []
            for p in range(Tk):
                s = 0.0
                for c in range(hd):
                    s += float(q[t, g, c]) * float(k[p, j, c])
                logits.append(s / math.sqrt(hd))
            mx = max(logits)
            ws = [math.exp(z - mx) for z in logits]
            tot = sum(ws)
            for c in range(hd):
                out[t, g, c] = sum(ws[p] * float(v[p, j, c]) for p in range(Tk)) / tot
    return out


def test_attention_matches_scalar_bruteforce():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((3, 4, 5))
    k = rng.standard_normal((7, 2, 5))
    v = rng.standard_normal((7, 2, 5))
    np.testing.assert_allclose(attention(q, k, v), _attention_scalar(q, k, v), rtol=1e-12, atol=1e-13)


def test_attention_single_key_returns_value():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((4, 2, 8))
    k = rng.standard_normal((1, 1, 8))
    v = rng.standard_normal((1, 1, 8))
    o = attention(q, k, v)
    for t in range(4):
        for g in range(2):
            np.testing.assert_array_equal(o[t, g], v[0, 0])


def test_attention_equal_keys_give_mean_value():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((2, 2, 6))
    k = np.repeat(rng.standard_normal((1, 1, 6)), 9, axis=0)
    v = rng.standard_normal((9, 1, 6))
    np.testing.assert_allclose(attention(q, k, v)[1, 1], v[:, 0].mean(axis=0), rtol=1e-13, atol=1e-14)


def test_attention_gqa_head_grouping():
    # 4 query heads over 2 KV heads: heads 0,1 read KV head 0; heads 2,3 read KV head 1.
    rng = np.random.default_rng(4)
    q = rng.standard_normal((3, 4, 4))
    k = rng.standard_normal((5, 2, 4))
    v = np.zeros((5, 2, 4))
    v[:, 0, :] = 1.0
    v[:, 1, :] = 2.0
    o = attention(q, k, v)
    np.testing.assert_allclose(o[:, :2], 1.0, rtol=0, atol=1e-14)
    np.testing.assert_allclose(o[:, 2:], 2.0, rtol=0, atol=1e-14)


def test_attention_scale_is_inverse_sqrt_head_dim():
    # Two keys whose logits differ by exactly sqrt(hd) * log(3): weights 3:1.
    hd = 16
    q = np.zeros((1, 1, hd)); q[0, 0, 0] = 1.0
    k = np.zeros((2, 1, hd)); k[0, 0, 0] = math.sqrt(hd) * math.log(3.0)
    v = np.zeros((2, 1, hd)); v[0, 0, 1] = 1.0; v[1, 0, 1] = 0.0
    o = attention(q, k, v)
    assert abs(o[0, 0, 1] - 0.75) < 1e-14


# ------------------------------------------------------------------ time embedding, norms, activations

def test_embedding_at_tau_zero():
    e = timestep_embedding(0.0, 128)
    np.testing.assert_array_equal(e[:64], 0.0)
    np.testing.assert_array_equal(e[64:], 1.0)


def test_embedding_pairs_on_unit_circle():
    for tau in [0.1, 0.37, 0.9]:
        e = timestep_embedding(tau, 64)
        np.testing.assert_allclose(e[:32] ** 2 + e[32:] ** 2, 1.0, atol=1e-14)


def test_embedding_frequencies_geometric():
    # tau small enough that every angle is in (0, pi/2): recover angles by atan2.
    tau, dim = 1e-4, 16
    e = timestep_embedding(tau, dim)
    half = dim // 2
    ang = np.arctan2(e[:half], e[half:])
    assert abs(ang[0] - 1000.0 * tau) < 1e-15          # first frequency is 1
    ratios = ang[1:] / ang[:-1]
    np.testing.assert_allclose(ratios, 10000.0 ** (-1.0 / half), rtol=1e-12)


def test_tau_grid_is_k_over_K():
    assert tau_grid(4) == [0.0, 0.25, 0.5, 0.75]
    g = tau_grid(10)
    assert len(g) == 10 and g[0] == 0.0 and abs(g[7] - 0.7) < 1e-7
    assert g[7] == float(np.float32(0.7))


def test_rmsnorm_constant_vector():
    eps = 1e-6
    for c in [-3.0, 0.01, 2.5]:
        h = np.full((1, 32), c)
        expect = math.copysign(1.0, c) / math.sqrt(1.0 + eps / (c * c))
        np.testing.assert_allclose(rms_norm(h, eps), expect, rtol=1e-14)


def test_rmsnorm_output_mean_square():
    rng = np.random.default_rng(5)
    h = rng.standard_normal((4, 100)) * 3.0
    eps = 1e-6
    y = rms_norm(h, eps)
    ms = (h * h).mean(axis=1)
    np.testing.assert_allclose((y * y).mean(axis=1), ms / (ms + eps), rtol=1e-13)


def test_gelu_tanh_against_erf_gelu():
    x = np.linspace(-6, 6, 2001)
    exact = np.array([0.5 * xi * (1.0 + math.erf(xi / math.sqrt(2.0))) for xi in x])
    assert np.max(np.abs(gelu_tanh(x) - exact)) < 1e-3       # tanh approximation error bound
    assert gelu_tanh(np.array([0.0]))[0] == 0.0
    assert abs(gelu_tanh(np.array([10.0]))[0] - 10.0) < 1e-12
    assert abs(gelu_tanh(np.array([-10.0]))[0]) < 1e-12


def test_gelu_tanh_pinned_values():
    """The tanh form's published cubic coefficient 0.044715 and its sqrt(2/pi)
    scale, pinned at points where they are fixed in closed form: at x = 1 the
    argument of tanh is sqrt(2/pi) * 1.044715, at x = 2 it is sqrt(2/pi) *
    (2 + 8 * 0.044715).  A coefficient off by 1e-9 moves these values by more
    than the tolerance.  The odd part of any x * (1 + tanh(odd(x))) / 2 is x / 2,
    so gelu(x) - gelu(-x) = x exactly in real arithmetic."""
    k = math.sqrt(2.0 / math.pi)
    assert abs(gelu_tanh(np.array([1.0]))[0] - 0.5 * (1.0 + math.tanh(k * 1.044715))) < 1e-15
    assert abs(gelu_tanh(np.array([2.0]))[0] - (1.0 + math.tanh(k * 2.35772))) < 1e-15
    assert abs(gelu_tanh(np.array([1.0]))[0] - 0.8411919906082768) < 1e-14   # 0.5 (1 + tanh(0.83356197))
    x = np.linspace(-5.0, 5.0, 101)
    np.testing.assert_allclose(gelu_tanh(x) - gelu_tanh(-x), x, rtol=0, atol=1e-14)


def test_silu_closed_forms():
    """SiLU(x) = x sigmoid(x): sigmoid(ln 3) = 3/4 gives SiLU(ln 3) = 0.75 ln 3,
    sigmoid(-ln 3) = 1/4; sigmoid(x) + sigmoid(-x) = 1 gives SiLU(x) - SiLU(-x) = x;
    SiLU(0) = 0 and SiLU(x) -> x, 0 at the two ends."""
    l3 = math.log(3.0)
    assert abs(silu(np.array([l3]))[0] - 0.75 * l3) < 1e-15
    assert abs(silu(np.array([-l3]))[0] + 0.25 * l3) < 1e-15
    assert silu(np.array([0.0]))[0] == 0.0
    x = np.linspace(-8.0, 8.0, 161)
    np.testing.assert_allclose(silu(x) - silu(-x), x, rtol=0, atol=1e-14)
    assert abs(silu(np.array([40.0]))[0] - 40.0) < 1e-12
    assert abs(silu(np.array([-40.0]))[0]) < 1e-12


# ------------------------------------------------------------------ Euler closed forms

def _zero_weights(shape):
    w = make_weights(shape, "fp32", seed=0)
    return {k: np.zeros_like(v) for k, v in w.items()}


def _grid_noise(rng, H, A, step=2.0 ** -8):
    return (np.round(rng.uniform(-4, 4, size=(H, A)) / step) * step).astype(np.float32)


@pytest.mark.parametrize("K", [1, 2, 4, 8])
def test_constant_velocity_exact_power_of_two_steps(K):
    w = _zero_weights(TINY_SHAPE)
    rng = np.random.default_rng(K)
    c = (np.round(rng.uniform(-2, 2, size=TINY_SHAPE.action_dim) * 16) / 16).astype(np.float32)
    w["b_out"] = c
    req = custom_request(TINY_SHAPE, "fp32", 5, 3, K, seed=11)
    req.noise = _grid_noise(rng, 3, TINY_SHAPE.action_dim)
    x = OracleModel(w, TINY_SHAPE).generate([req])[0]
    np.testing.assert_array_equal(x, req.noise.astype(np.float64) + c)


@pytest.mark.parametrize("K", [3, 5, 10])
def test_constant_velocity_other_steps(K):
    w = _zero_weights(TINY_SHAPE)
    c = np.linspace(-1, 1, TINY_SHAPE.action_dim).astype(np.float32)
    w["b_out"] = c
    req = custom_request(TINY_SHAPE, "fp32", 4, 2, K, seed=12)
    x = OracleModel(w, TINY_SHAPE).generate([req])[0]
    np.testing.assert_allclose(x, req.noise.astype(np.float64) + c, rtol=0, atol=1e-14)


def test_advance_constant_velocity_partial_steps():
    # steps k0 .. k1-1 of K under v = c add c (k1 - k0) / K
    w = _zero_weights(TINY_SHAPE)
    rng = np.random.default_rng(21)
    c = (np.round(rng.uniform(-2, 2, size=TINY_SHAPE.action_dim) * 16) / 16).astype(np.float32)
    w["b_out"] = c
    om = OracleModel(w, TINY_SHAPE)
    req = custom_request(TINY_SHAPE, "fp32", 6, 3, 8, seed=22)
    x0 = _grid_noise(rng, 3, TINY_SHAPE.action_dim).astype(np.float64)
    pk, pv = req.prefix_f32("k"), req.prefix_f32("v")
    for k0, k1 in [(0, 3), (3, 8), (5, 6)]:
        np.testing.assert_array_equal(om.advance(x0, 8, k0, k1, pk, pv), x0 + c * (k1 - k0) / 8.0)


def test_advance_in_pieces_equals_one_shot():
    # regrouping the Euler steps (as step-level batching does) reproduces the
    # whole chunk exactly: each piece keeps its own flow times k / K
    w = make_weights(TINY_SHAPE, "fp32", seed=3)
    om = OracleModel(w, TINY_SHAPE)
    req = custom_request(TINY_SHAPE, "fp32", 20, 4, 5, seed=23)
    pk, pv = req.prefix_f32("k"), req.prefix_f32("v")
    whole = om.generate_chunk(req.noise, 5, pk, pv)
    x = req.noise.astype(np.float64)
    for k0, k1 in [(0, 2), (2, 3), (3, 5)]:
        x = om.advance(x, 5, k0, k1, pk, pv)
    np.testing.assert_array_equal(x, whole)


def test_zero_velocity_keeps_noise():
    w = make_weights(TINY_SHAPE, "fp32", seed=0)
    w["w_out"][:] = 0.0
    w["b_out"][:] = 0.0
    req = custom_request(TINY_SHAPE, "fp32", 17, 5, 4, seed=13)
    x = OracleModel(w, TINY_SHAPE).generate([req])[0]
    np.testing.assert_array_equal(x, req.noise.astype(np.float64))


def test_zero_gates_closed_form():
    """With every modulation projection zero, each block is the identity and the
    final norm is unmodulated, so v = RMSNorm(x W_in + b_in) W_out + b_out."""
    rng = np.random.default_rng(6)
    w = make_weights(TINY_SHAPE, "fp32", seed=0)
    for k in ["w_mod", "b_mod", "w_fmod", "b_fmod"]:
        w[k][:] = 0.0
    w["b_in"] = rng.standard_normal(w["b_in"].shape).astype(np.float32) * 0.1
    w["b_out"] = rng.standard_normal(w["b_out"].shape).astype(np.float32) * 0.1
    req = custom_request(TINY_SHAPE, "fp32", 9, 4, 1, seed=14)
    x0 = req.noise.astype(np.float64)
    h = x0 @ w["w_in"].astype(np.float64) + w["b_in"]
    h = h / np.sqrt((h * h).mean(axis=1, keepdims=True) + 1e-6)
    v = h @ w["w_out"].astype(np.float64) + w["b_out"]
    x = OracleModel(w, TINY_SHAPE).generate([req])[0]
    np.testing.assert_allclose(x, x0 + v, rtol=1e-12, atol=1e-13)


# ------------------------------------------------------------------ whole forward, scalar brute force

def _scalar_forward(w, sh, noise, K, pk, pv, layout=0):
    """The whole generate loop on nested Python lists and floats.  layout 1:
    even layers see only the prefix keys, odd layers only the action keys."""
    d, nq, nkv, hd, A = sh.d_model, sh.n_q_heads, sh.n_kv_heads, sh.head_dim, sh.action_dim
    H = len(noise)
    W = {k: v.astype(np.float64).tolist() for k, v in w.items()}

    def vecmat(x, M):            # x: [n], M: [n][m]
        return [sum(x[i] * M[i][j] for i in range(len(x))) for j in range(len(M[0]))]

    def sig(z):
        return 1.0 / (1.0 + math.exp(-z))

    def norm(row, shift, scale):
        ms = sum(z * z for z in row) / len(row)
        r = 1.0 / math.sqrt(ms + sh.rms_eps)
        return [row[i] * r * (1.0 + scale[i]) + shift[i] for i in range(len(row))]

    x = [[float(z) for z in row] for row in noise]
    for k in range(K):
        tau = float(np.float32(k) / np.float32(K))
        half = sh.time_emb_dim // 2
        ang = [1000.0 * tau * 10000.0 ** (-i / half) for i in range(half)]
        e = [math.sin(a) for a in ang] + [math.cos(a) for a in ang]
        t1 = [z * sig(z) for z in [a + b for a, b in zip(vecmat(e, W["w_t1"]), W["b_t1"])]]
        c = [a + b for a, b in zip(vecmat(t1, W["w_t2"]), W["b_t2"])]
        s = [z * sig(z) for z in c]
        h = [[a + b for a, b in zip(vecmat(x[t], W["w_in"]), W["b_in"])] for t in range(H)]
        for l in range(sh.n_layers):
            m = [a + b for a, b in zip(vecmat(s, W["w_mod"][l]), W["b_mod"][l])]
            sa, ca, ga, sm, cm, gm = [m[i * d:(i + 1) * d] for i in range(6)]
            u = [norm(h[t], sa, ca) for t in range(H)]
            qkv = [vecmat(u[t], W["w_qkv"][l]) for t in range(H)]
            o = [[0.0] * (nq * hd) for _ in range(H)]
            for t in range(H):
                for g in range(nq):
                    j = g // (nq // nkv)
                    qv = qkv[t][g * hd:(g + 1) * hd]
                    pre_k = [list(map(float, pk[l][p][j])) for p in range(len(pk[l]))]
                    act_k = [qkv[tt][nq * hd + j * hd: nq * hd + (j + 1) * hd] for tt in range(H)]
                    pre_v = [list(map(float, pv[l][p][j])) for p in range(len(pv[l]))]
                    act_v = [qkv[tt][(nq + nkv) * hd + j * hd: (nq + nkv) * hd + (j + 1) * hd]
                             for tt in range(H)]
                    if layout == 1 and l % 2 == 0:
                        keys, vals = pre_k, pre_v
                    elif layout == 1:
                        keys, vals = act_k, act_v
                    else:
                        keys, vals = pre_k + act_k, pre_v + act_v
                    lg = [sum(qv[c2] * kk[c2] for c2 in range(hd)) / math.sqrt(hd) for kk in keys]
                    mx = max(lg)
                    ws = [math.exp(z - mx) for z in lg]
                    tot = sum(ws)
                    for c2 in range(hd):
                        o[t][g * hd + c2] = sum(ws[p] * vals[p][c2] for p in range(len(keys))) / tot
            for t in range(H):
                a = vecmat(o[t], W["w_o"][l])
                h[t] = [h[t][i] + ga[i] * a[i] for i in range(d)]
            u = [norm(h[t], sm, cm) for t in range(H)]
            for t in range(H):
                up = vecmat(u[t], W["w_up"][l])
                gl = [0.5 * z * (1.0 + math.tanh(math.sqrt(2.0 / math.pi) * (z + 0.044715 * z ** 3)))
                      for z in up]
                dn = vecmat(gl, W["w_down"][l])
                h[t] = [h[t][i] + gm[i] * dn[i] for i in range(d)]
        fm = [a + b for a, b in zip(vecmat(s, W["w_fmod"]), W["b_fmod"])]
        sf, cf = fm[:d], fm[d:]
        for t in range(H):
            vel = [a + b for a, b in zip(vecmat(norm(h[t], sf, cf), W["w_out"]), W["b_out"])]
            x[t] = [x[t][i] + (1.0 / K) * vel[i] for i in range(A)]
    return np.array(x)


@pytest.mark.parametrize("nkv", [1, 2])
def test_whole_forward_matches_scalar_bruteforce(nkv):
    sh = dataclasses.replace(MICRO, n_kv_heads=nkv)
    w = make_weights(sh, "fp32", seed=3, std=0.3)   # large weights: every term matters
    rng = np.random.default_rng(7)
    for k in ["b_in", "b_t1", "b_t2", "b_mod", "b_fmod", "b_out"]:
        w[k] = (rng.standard_normal(w[k].shape) * 0.2).astype(np.float32)
    req = custom_request(sh, "fp32", 3, 2, 3, seed=15)
    ref = _scalar_forward(w, sh, req.noise, req.steps, req.prefix_k, req.prefix_v)
    got = OracleModel(w, sh).generate([req])[0]
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("P", [1, 3])
def test_alternating_layout_matches_scalar_bruteforce(P):
    sh = dataclasses.replace(MICRO, n_layers=4, attention_layout=1)
    w = make_weights(sh, "fp32", seed=4, std=0.3)
    rng = np.random.default_rng(8)
    for k in ["b_in", "b_t1", "b_t2", "b_mod", "b_fmod", "b_out"]:
        w[k] = (rng.standard_normal(w[k].shape) * 0.2).astype(np.float32)
    req = custom_request(sh, "fp32", P, 3, 2, seed=16)
    ref = _scalar_forward(w, sh, req.noise, req.steps, req.prefix_k, req.prefix_v, layout=1)
    got = OracleModel(w, sh).generate([req])[0]
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)
    joint = OracleModel(w, dataclasses.replace(sh, attention_layout=0)).generate([req])[0]
    assert np.abs(joint - got).max() > 1e-6          # the layouts differ


def test_alternating_layout_reads_prefix_in_even_layers_only():
    sh = dataclasses.replace(TINY_SHAPE, attention_layout=1)
    w = make_weights(sh, "fp32", seed=0)
    d = sh.d_model
    w["w_down"][:] = 0.0
    w["b_mod"][:, 2 * d:3 * d] = 1.0                 # attention-isolating variant
    r = custom_request(sh, "fp32", 40, 8, 4, seed=40)
    m = OracleModel(w, sh)
    base = m.generate([r])[0]
    odd = dataclasses.replace(r, prefix_k=r.prefix_k.copy(), prefix_v=r.prefix_v.copy())
    odd.prefix_k[1::2] = np.random.default_rng(1).standard_normal(odd.prefix_k[1::2].shape)
    odd.prefix_v[1::2] = 0.0
    np.testing.assert_array_equal(m.generate([odd])[0], base)
    even = dataclasses.replace(r, prefix_k=r.prefix_k.copy(), prefix_v=r.prefix_v.copy())
    even.prefix_v[0::2] *= -1.0
    assert np.abs(m.generate([even])[0] - base).max() > 1e-3


# ------------------------------------------------------------------ invariants

def test_batch_and_permutation_invariance():
    w = make_weights(TINY_SHAPE, "fp32", seed=0)
    reqs = [custom_request(TINY_SHAPE, "fp32", P, H, K, seed=20 + i)
            for i, (P, H, K) in enumerate([(64, 8, 4), (0, 3, 2), (96, 5, 5)])]
    m = OracleModel(w, TINY_SHAPE)
    batched = m.generate(reqs)
    alone = [m.generate([r])[0] for r in reqs]
    perm = m.generate([reqs[2], reqs[0], reqs[1]])
    for a, b in zip(batched, alone):
        np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(perm[0], batched[2])
    np.testing.assert_array_equal(perm[1], batched[0])


def test_prefix_swap_visible_in_attention_isolating_variant():
    """With the MLP removed and the attention gate biased to one, swapping two
    requests' prefix caches must move the result far beyond a 1e-2 gate: the
    end-to-end comparison can see attention mistakes."""
    w = make_weights(TINY_SHAPE, "fp32", seed=0)
    d = TINY_SHAPE.d_model
    w["w_down"][:] = 0.0
    w["b_mod"][:, 2 * d:3 * d] = 1.0
    a = custom_request(TINY_SHAPE, "fp32", 64, 8, 4, seed=30)
    b = custom_request(TINY_SHAPE, "fp32", 96, 8, 4, seed=31)
    m = OracleModel(w, TINY_SHAPE)
    xa = m.generate([a])[0]
    a.prefix_k, a.prefix_v = b.prefix_k, b.prefix_v
    xs = m.generate([a])[0]
    disp = xa - a.noise
    assert np.linalg.norm(xs - xa) / np.linalg.norm(disp) > 5e-2
