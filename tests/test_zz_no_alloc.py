"""GPU test of the allocation-free attention entry point (rosa_attention_noalloc)
against the handle-based one (rosa_debug_attention) on the same inputs, two
calls in a row (the second with fewer requests), plus sampled requests against
the oracle's attention."""
import dataclasses

import numpy as np
import pytest

from oracle import attention as oracle_attention
from synthetic import PI0_SHAPE, TINY_SHAPE, bits_to_f32, weight_shapes
from tests.helpers import rel_l2

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

# pi0 attention width (8 query heads over one 256-wide KV head) with two layers
SHAPE = dataclasses.replace(PI0_SHAPE, n_layers=2)


def _host(t):
    if t.dtype == torch.bfloat16:
        return bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16))
    return t.cpu().numpy()


def _case(shape, dtype, specs, seed):
    from paper_2607_01088_amd import rosa
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    L, nq, nkv, hd = shape.n_layers, shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    keep, structs = [], []
    dummy = torch.zeros(64, dtype=torch.float32, device="cuda")
    for P, H in specs:
        k = torch.randn((L, max(P, 1), nkv, hd), device="cuda", dtype=tdt, generator=g)
        v = torch.randn((L, max(P, 1), nkv, hd), device="cuda", dtype=tdt, generator=g)
        keep.append((k, v))
        structs.append(rosa.request_struct(k if P else None, v if P else None, dummy, dummy, P, H, 1))
    M = sum(H for _, H in specs)
    qkv = torch.randn((M, (nq + 2 * nkv) * hd), device="cuda", dtype=tdt, generator=g)
    qkv[:, : nq * hd] *= 0.25
    return keep, structs, qkv


def _oracle_one(shape, qkv_h, keep, specs, i, layer):
    nq, nkv, hd = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    row = sum(H for _, H in specs[:i])
    P, H = specs[i]
    rows = qkv_h[row:row + H].astype(np.float64)
    q = rows[:, : nq * hd].reshape(H, nq, hd)
    ka = rows[:, nq * hd:(nq + nkv) * hd].reshape(H, nkv, hd)
    va = rows[:, (nq + nkv) * hd:].reshape(H, nkv, hd)
    k = _host(keep[i][0][layer, :P]).astype(np.float64)
    v = _host(keep[i][1][layer, :P]).astype(np.float64)
    return oracle_attention(q, np.concatenate([k, ka]), np.concatenate([v, va])).reshape(H, nq * hd), row


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_noalloc_attention_matches_handle_attention(dtype):
    from paper_2607_01088_amd import rosa
    shape = SHAPE if dtype == "bf16" else TINY_SHAPE
    w = {k: np.zeros(s, np.float32) for k, s in weight_shapes(shape).items()}
    rng = np.random.default_rng(21)
    # call 1: enough query blocks that neither entry point splits keys
    # (bitwise equal); call 2: fewer requests, key ranges split over items
    big = [(int(rng.integers(0, 1500)), int(rng.integers(1, 51))) for _ in range(130)]
    big[0], big[1] = (0, 50), (1, 1)
    small = [(1400, 50), (700, 16), (33, 5), (1, 3)]
    cap = rosa.capacity(len(big), 50, sum(H for _, H in big), 10, sum(P for P, _ in big))
    e = rosa.ActionExpert(shape, dtype, w, cap)
    try:
        for call, specs in enumerate([big, small]):
            keep, structs, qkv = _case(shape, dtype, specs, seed=100 + call)
            layer = shape.n_layers - 1
            M = qkv.shape[0]
            o_ref = torch.full((M, shape.n_q_heads * shape.head_dim), float("nan"), dtype=qkv.dtype, device="cuda")
            o_new = torch.full_like(o_ref, float("nan"))
            e.attention(structs, layer, qkv, o_ref)
            st = rosa.attention_noalloc(shape, dtype, structs, layer, qkv, o_new)
            assert st == rosa.ROSA_OK, rosa.last_error_global()
            torch.cuda.synchronize()
            ref, got = _host(o_ref), _host(o_new)
            assert np.isfinite(got).all()
            split_plan = rosa.plan(shape, dtype, cap, structs)[4][3] > 0
            print(f"{dtype} call {call}: {len(specs)} requests, handle path splits keys: {split_plan}", flush=True)
            if not split_plan:
                assert np.array_equal(got, ref)
            row = 0
            for i, (P, H) in enumerate(specs):
                err = rel_l2(got[row:row + H], ref[row:row + H])
                assert err <= (1e-2 if dtype == "bf16" else 1e-5), (call, i, P, H, err)
                row += H
            qkv_h = _host(qkv)
            for i in sorted({0, 1, len(specs) - 1, int(np.argmax([P for P, _ in specs]))}):
                want, r0 = _oracle_one(shape, qkv_h, keep, specs, i, layer)
                err = rel_l2(got[r0:r0 + specs[i][1]], want)
                assert err <= (1e-2 if dtype == "bf16" else 1e-5), (call, i, err)
    finally:
        e.close()


def test_noalloc_attention_rejects_beyond_limits():
    from paper_2607_01088_amd import rosa
    shape = SHAPE
    qkv = torch.zeros((2, (shape.n_q_heads + 2) * shape.head_dim), dtype=torch.bfloat16, device="cuda")
    o = torch.zeros((2, shape.n_q_heads * shape.head_dim), dtype=torch.bfloat16, device="cuda")
    dummy = torch.zeros(64, dtype=torch.float32, device="cuda")
    reqs = [rosa.request_struct(None, None, dummy, dummy, 0, 1, 1)] * 1025
    assert rosa.attention_noalloc(shape, "bf16", reqs, 0, qkv, o) == rosa.ROSA_E_CAPACITY
    assert "1024" in rosa.last_error_global()
    assert rosa.attention_noalloc(shape, "bf16", reqs[:2], 2, qkv, o) == rosa.ROSA_E_INVALID
    bad = [rosa.request_struct(None, None, dummy, dummy, 0, 0, 1)]
    assert rosa.attention_noalloc(shape, "bf16", bad, 0, qkv, o) == rosa.ROSA_E_INVALID
    assert rosa.attention_noalloc(shape, "bf16", [], 0, qkv, o) == rosa.ROSA_OK
