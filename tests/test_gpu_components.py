"""GPU parity of the library's components against the CPU oracle, through the
C ABI's component entry points (rosa_debug.h)."""
import math

import numpy as np
import pytest

from oracle import OracleModel, attention as oracle_attention, gelu_tanh
from synthetic import PI0_SHAPE, TINY_SHAPE, bf16_round, bits_to_f32, bf16_bits
from tests.helpers import cached_weights, rel_l2

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _expert(shape, dtype, max_requests=8, max_horizon=50, max_tokens=2048, max_steps=10,
            max_prefix=1 << 16):
    from paper_2607_01088_amd import rosa
    w = cached_weights(shape, dtype)
    cap = rosa.capacity(max_requests, max_horizon, max_tokens, max_steps, max_prefix)
    return rosa.ActionExpert(shape, dtype, w, cap), w


@pytest.fixture(scope="module")
def tiny_fp32():
    e, w = _expert(TINY_SHAPE, "fp32")
    yield e, w
    e.close()


@pytest.fixture(scope="module")
def tiny_bf16():
    e, w = _expert(TINY_SHAPE, "bf16")
    yield e, w
    e.close()


@pytest.fixture(scope="module")
def hd64_bf16():
    from tests.helpers import HD64_SHAPE
    e, w = _expert(HD64_SHAPE, "bf16")
    yield e, w
    e.close()


@pytest.fixture(scope="module")
def hd128_bf16():
    from tests.helpers import HD128_SHAPE
    e, w = _expert(HD128_SHAPE, "bf16")
    yield e, w
    e.close()


@pytest.fixture(scope="module")
def pi0_bf16():
    e, w = _expert(PI0_SHAPE, "bf16", max_requests=160, max_tokens=160 * 50)
    yield e, w
    e.close()


def _tdev(a, dtype):
    if dtype == "bf16":
        return torch.from_numpy(bf16_bits(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def _thost(t):
    if t.dtype == torch.bfloat16:
        return bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16))
    return t.cpu().numpy()


# ------------------------------------------------------------------ time conditioning

@pytest.mark.parametrize("which", ["tiny_fp32", "tiny_bf16", "pi0_bf16"])
def test_time_conditioning_matches_oracle(which, request):
    e, w = request.getfixturevalue(which)
    sh = e.shape
    taus = sorted({float(np.float32(k) / np.float32(K)) for K in (4, 5, 10) for k in range(K)})
    stride = sh.n_layers * 6 * sh.d_model + 2 * sh.d_model
    out = torch.empty((len(taus), stride), dtype=torch.float32, device="cuda")
    e.time_conditioning(taus, out)
    got = out.cpu().numpy()
    om = OracleModel(w, sh)
    for i, tau in enumerate(taus):
        s = om.time_condition(tau)
        ref = np.concatenate([np.concatenate(om.block_modulation(s, l)) for l in range(sh.n_layers)]
                             + [np.concatenate(om.final_modulation(s))])
        assert rel_l2(got[i], ref) < 1e-5, (tau, rel_l2(got[i], ref))


# ------------------------------------------------------------------ projections

@pytest.mark.parametrize("which", ["tiny_fp32", "tiny_bf16", "pi0_bf16"])
@pytest.mark.parametrize("proj", [0, 1, 2, 3])
@pytest.mark.parametrize("M", [1, 50, 129, 256, 257, 1600])
def test_projection_matches_float64(which, proj, M, request):
    e, w = request.getfixturevalue(which)
    sh, dtype = e.shape, e.dtype
    if M > e.cap.max_action_tokens:
        pytest.skip("above capacity")
    layer = sh.n_layers - 1
    rng = np.random.default_rng(100 + proj + M)
    K_in = {0: sh.d_model, 1: sh.n_q_heads * sh.head_dim, 2: sh.d_model, 3: sh.d_mlp}[proj]
    W = {0: w["w_qkv"], 1: w["w_o"], 2: w["w_up"], 3: w["w_down"]}[proj][layer].astype(np.float64)
    a = rng.standard_normal((M, K_in)).astype(np.float32)
    if dtype == "bf16":
        a = bf16_round(a)
    acc = a.astype(np.float64) @ W
    a_dev = _tdev(a, dtype)
    tol = 1e-5 if dtype == "fp32" else 1e-2
    if proj in (0, 2):
        out = torch.empty((M, W.shape[1]), dtype=a_dev.dtype, device="cuda")
        e.gemm(proj, layer, a_dev, M, out)
        ref = acc if proj == 0 else gelu_tanh(acc)
        got = _thost(out)
        assert rel_l2(got, ref) < (1e-5 if dtype == "fp32" else 4e-3)
    else:
        h0 = rng.standard_normal((M, sh.d_model)).astype(np.float32)
        gate = rng.standard_normal((M, sh.d_model)).astype(np.float32)
        h = torch.from_numpy(h0).cuda()
        e.gemm(proj, layer, a_dev, M, h, torch.from_numpy(gate).cuda())
        got = h.cpu().numpy().astype(np.float64) - h0
        assert rel_l2(got, gate * acc) < (1e-5 if dtype == "fp32" else 1e-5), tol


@pytest.mark.parametrize("which,M", [("tiny_bf16", 129), ("pi0_bf16", 50), ("pi0_bf16", 1600)])
@pytest.mark.parametrize("proj", [0, 1, 2, 3])
def test_projection_each_block_config(which, M, proj, request):
    """Every bf16 block configuration against float64, and bitwise equal to
    the others (the same MFMA sequence computes each output)."""
    e, w = request.getfixturevalue(which)
    sh = e.shape
    if M > e.cap.max_action_tokens:
        pytest.skip("above capacity")
    layer = 0
    rng = np.random.default_rng(7 + proj + M)
    K_in = {0: sh.d_model, 1: sh.n_q_heads * sh.head_dim, 2: sh.d_model, 3: sh.d_mlp}[proj]
    W = {0: w["w_qkv"], 1: w["w_o"], 2: w["w_up"], 3: w["w_down"]}[proj][layer].astype(np.float64)
    a = bf16_round(rng.standard_normal((M, K_in)).astype(np.float32))
    acc = a.astype(np.float64) @ W
    a_dev = _tdev(a, "bf16")
    h0 = rng.standard_normal((M, sh.d_model)).astype(np.float32)
    gate = torch.from_numpy(rng.standard_normal((M, sh.d_model)).astype(np.float32)).cuda()
    outs = []
    n_cfg = e.gemm_config(-1)
    try:
        for cfg in range(n_cfg):
            e.gemm_config(cfg)
            if proj in (0, 2):
                out = torch.full((M, W.shape[1]), float("nan"), dtype=a_dev.dtype, device="cuda")
                e.gemm(proj, layer, a_dev, M, out)
                got = _thost(out)
                ref = acc if proj == 0 else gelu_tanh(acc)
                err = rel_l2(got, ref)
                assert err < 4e-3, (cfg, err)
            else:
                h = torch.from_numpy(h0).cuda()
                e.gemm(proj, layer, a_dev, M, h, gate)
                got = h.cpu().numpy()
                err = rel_l2(got.astype(np.float64) - h0, gate.cpu().numpy() * acc)
                assert err < 1e-5, (cfg, err)
            outs.append(got)
    finally:
        e.gemm_config(-1)
    for cfg in range(1, n_cfg):
        assert np.array_equal(outs[cfg], outs[0]), cfg


# ------------------------------------------------------------------ attention

def _attn_case(e, shapes, seed, fill_q=None, tags=None):
    """Random (or tagged) attention inputs for requests of (P, H); returns the
    device buffers, request structs and host copies."""
    from paper_2607_01088_amd import rosa
    sh, dtype = e.shape, e.dtype
    L, nq, nkv, hd = sh.n_layers, sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    Q = (nq + 2 * nkv) * hd
    rng = np.random.default_rng(seed)
    M = sum(H for _, H in shapes)
    guard = 8
    qkv = rng.standard_normal((M + guard, Q)).astype(np.float32)
    qkv[:, : nq * hd] *= 0.25 if fill_q is None else 1.0
    if fill_q is not None:
        qkv[:, : nq * hd] = fill_q
    qkv[M:] = np.nan                                  # rows past the batch are poison
    if dtype == "bf16":
        qkv = bf16_round(qkv)
    keep, structs, host = [], [], []
    row = 0
    for i, (P, H) in enumerate(shapes):
        k = rng.standard_normal((L, P + guard, nkv, hd)).astype(np.float32)
        v = rng.standard_normal((L, P + guard, nkv, hd)).astype(np.float32)
        if tags is not None:
            # one tag per request, or one per (request, KV head)
            t = np.broadcast_to(np.asarray(tags[i], dtype=np.float32), (nkv,))
            for j in range(nkv):
                v[:, :, j, :] = t[j]
                qkv[row:row + H, (nq + nkv + j) * hd:(nq + nkv + j + 1) * hd] = t[j]
        k[:, P:] = np.nan                                # guard tokens after each prefix
        v[:, P:] = np.nan
        if dtype == "bf16":
            k, v = bf16_round(k), bf16_round(v)
        # the library's layout is [L][P][n_kv][hd] with layer stride P: drop the guard per layer
        kd = _tdev(np.ascontiguousarray(k[:, :P]).reshape(-1), dtype) if P > 0 else None
        vd = _tdev(np.ascontiguousarray(v[:, :P]).reshape(-1), dtype) if P > 0 else None
        if P > 0:
            # re-append a NaN guard after the whole buffer
            kd = torch.cat([kd, torch.full((guard * nkv * hd,), float("nan"), dtype=kd.dtype, device="cuda")])
            vd = torch.cat([vd, torch.full((guard * nkv * hd,), float("nan"), dtype=vd.dtype, device="cuda")])
        keep += [kd, vd]
        structs.append(rosa.request_struct(kd, vd, 0x1000, 0x1000, P, H, 1))
        host.append((k[:, :P], v[:, :P], row, H))
        row += H
    qkv_d = _tdev(qkv, dtype)
    o = torch.full((M + guard, nq * hd), float("nan"), dtype=qkv_d.dtype, device="cuda")
    return qkv, qkv_d, o, structs, host, keep


def _oracle_attn(sh, qkv, host, layer):
    nq, nkv, hd = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    outs = []
    for k, v, row, H in host:
        rows = qkv[row:row + H].astype(np.float64)
        q = rows[:, : nq * hd].reshape(H, nq, hd)
        ka = rows[:, nq * hd:(nq + nkv) * hd].reshape(H, nkv, hd)
        va = rows[:, (nq + nkv) * hd:].reshape(H, nkv, hd)
        kf = np.concatenate([k[layer].astype(np.float64), ka])
        vf = np.concatenate([v[layer].astype(np.float64), va])
        outs.append(oracle_attention(q, kf, vf).reshape(H, nq * hd))
    return outs


ATTN_CASES = {
    "tiny": [(64, 8), (96, 8), (0, 3), (1, 1), (65, 5)],
    "pi0_ragged": [(816, 50), (63, 16), (64, 1), (65, 50), (0, 16), (2048, 50), (1, 16)],
    # head_dim 64 / 128 shapes: several 32-key tiles, ragged tails, P = 0 and 1,
    # one and several query blocks, a prefix long enough to split over items
    "head_dims": [(97, 17), (0, 5), (1, 1), (64, 33), (300, 50), (1500, 50), (31, 16)],
}


@pytest.mark.parametrize("which,case", [("tiny_fp32", "tiny"), ("tiny_bf16", "tiny"),
                                        ("pi0_bf16", "pi0_ragged")])
@pytest.mark.parametrize("layer_sel", ["first", "last"])
def test_attention_matches_oracle(which, case, layer_sel, request):
    e, _ = request.getfixturevalue(which)
    sh = e.shape
    layer = 0 if layer_sel == "first" else sh.n_layers - 1
    shapes = ATTN_CASES[case]
    qkv, qkv_d, o, structs, host, keep = _attn_case(e, shapes, seed=7)
    e.attention(structs, layer, qkv_d, o)
    got = _thost(o)
    refs = _oracle_attn(sh, qkv, host, layer)
    tol = 1e-5 if e.dtype == "fp32" else 1e-2
    M = sum(H for _, H in shapes)
    assert np.isnan(got[M:]).all()                      # nothing written past the batch
    for (P, H), (_, _, row, _), ref in zip(shapes, host, refs):
        err = rel_l2(got[row:row + H], ref)
        assert err < tol, (P, H, err)


@pytest.mark.parametrize("which", ["tiny_bf16", "pi0_bf16"])
def test_attention_score_far_above_first_tile(which, request):
    """One key in a late tile scores far above every key of the first tile
    (2^130 for head_dim 32, 2^208 for 256 in exp2 units): a single pass
    referenced to the first tile's max would overflow fp32, so the kernel must
    take its second pass and match the oracle's near one-hot softmax."""
    e, _ = request.getfixturevalue(which)
    sh = e.shape
    nq, nkv, hd = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    amp = 4.0 if hd == 32 else 3.0
    P, H, hot = 200, 4, 150
    qkv, qkv_d, o, structs, host, keep = _attn_case(e, [(P, H)], seed=3, fill_q=amp)
    k, v, row, _ = host[0]
    k[:] *= 0.01
    k[:, hot] = amp
    if e.dtype == "bf16":
        k[:] = bf16_round(k)
    kd, vd = keep[0], keep[1]
    kd[: k.size].copy_(_tdev(np.ascontiguousarray(k).reshape(-1), e.dtype))
    e.attention(structs, 1, qkv_d, o)
    got = _thost(o)[row:row + H]
    ref = _oracle_attn(sh, qkv, [(k, v, row, H)], 1)[0]
    assert np.isfinite(got).all()
    assert rel_l2(got, ref) < 1e-2
    # the softmax is one-hot on the hot key: every head returns its value row
    assert rel_l2(got.reshape(H, nq, hd), np.broadcast_to(v[1, hot, 0].astype(np.float64), (H, nq, hd))) < 1e-2


def test_attention_unsplit_batch(pi0_bf16):
    """A batch with enough query blocks to fill the GPU runs every request's
    keys in one work item (no partials, no merge); sampled requests match."""
    from paper_2607_01088_amd import rosa
    e, _ = pi0_bf16
    rng = np.random.default_rng(5)
    shapes = [(int(rng.integers(0, 300)), 50) for _ in range(130)]
    qkv, qkv_d, o, structs, host, keep = _attn_case(e, shapes, seed=12)
    st, _, _, _, counts = rosa.plan(e.shape, e.dtype, e.cap, structs)
    assert st == 0 and counts[3] == 0 and counts[1] == 130 * 4
    e.attention(structs, 0, qkv_d, o)
    got = _thost(o)
    refs = _oracle_attn(e.shape, qkv, host, 0)
    for i in [0, 1, 64, 127, 129]:
        P, H = shapes[i]
        row = host[i][2]
        assert rel_l2(got[row:row + H], refs[i]) < 1e-2, (i, P)


@pytest.mark.parametrize("which,case", [("tiny_fp32", "tiny"), ("tiny_bf16", "tiny"),
                                        ("pi0_bf16", "pi0_ragged")])
def test_attention_tag_bitwise(which, case, request):
    """Q = 0 and every value of request r equal to t_r: each output row of r is
    t_r exactly (uniform weights, exact sums), and NaN guards after every prefix
    and after the batch show any over-read."""
    e, _ = request.getfixturevalue(which)
    shapes = ATTN_CASES[case]
    tags = [float(i + 1) for i in range(len(shapes))]
    qkv, qkv_d, o, structs, host, keep = _attn_case(e, shapes, seed=3, fill_q=0.0, tags=tags)
    e.attention(structs, e.shape.n_layers - 1, qkv_d, o)
    got = _thost(o)
    for (P, H), (_, _, row, _), t in zip(shapes, host, tags):
        assert np.array_equal(got[row:row + H], np.full_like(got[row:row + H], t)), (P, H)


@pytest.mark.parametrize("which", ["hd64_bf16", "hd128_bf16"])
@pytest.mark.parametrize("layer_sel", ["first", "last"])
def test_attention_head_dims_matches_oracle(which, layer_sel, request):
    """The bf16 attention kernel at head_dim 64 (two query heads per KV head,
    two KV heads) and 128 (three KV heads, one query head each), element by
    element against the oracle; nothing is written past the batch."""
    e, _ = request.getfixturevalue(which)
    sh = e.shape
    layer = 0 if layer_sel == "first" else sh.n_layers - 1
    shapes = ATTN_CASES["head_dims"]
    qkv, qkv_d, o, structs, host, keep = _attn_case(e, shapes, seed=11)
    e.attention(structs, layer, qkv_d, o)
    got = _thost(o)
    refs = _oracle_attn(sh, qkv, host, layer)
    M = sum(H for _, H in shapes)
    assert np.isnan(got[M:]).all()
    for (P, H), (_, _, row, _), ref in zip(shapes, host, refs):
        err = rel_l2(got[row:row + H], ref)
        assert err < 1e-2, (P, H, err)


@pytest.mark.parametrize("which", ["hd64_bf16", "hd128_bf16"])
def test_attention_head_dims_tag_bitwise(which, request):
    """Q = 0 and every value of KV head j of request r equal to its own tag
    t_rj: each output of query head g is exactly t_r(g // G), so a wrong KV
    head, request or row offset fails bitwise."""
    e, _ = request.getfixturevalue(which)
    sh = e.shape
    nq, nkv, hd = sh.n_q_heads, sh.n_kv_heads, sh.head_dim
    G = nq // nkv
    shapes = ATTN_CASES["head_dims"]
    tags = [[float(4 * i + j + 1) for j in range(nkv)] for i in range(len(shapes))]
    qkv, qkv_d, o, structs, host, keep = _attn_case(e, shapes, seed=3, fill_q=0.0, tags=tags)
    e.attention(structs, sh.n_layers - 1, qkv_d, o)
    got = _thost(o)
    for (P, H), (_, _, row, _), t in zip(shapes, host, tags):
        want = np.empty((H, nq, hd), dtype=np.float32)
        for g in range(nq):
            want[:, g, :] = t[g // G]
        assert np.array_equal(got[row:row + H].reshape(H, nq, hd), want), (P, H)
