"""GPU parity of the alternating attention layout (a GR00T-style DiT head:
even layers cross-attend to the request's prefix, odd layers self-attend to
its action tokens; Sec. 2.2.1) against the oracle: the attention component per
layer kind, whole calls in fp32 and bf16 (small batches whose prefix keys are
split over work items, and a 160-request batch run in two lanes), and the
validation of requests without a prefix."""
import dataclasses

import numpy as np
import pytest

from oracle import OracleModel, attention as oracle_attention
from synthetic import PI0_ALT_SHAPE, PRESETS, TINY_ALT_SHAPE, custom_request, make_requests
from tests.helpers import cached_weights, rel_l2
from tests.test_gpu_components import _attn_case, _thost

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _rosa():
    from paper_2607_01088_amd import rosa
    return rosa


def _expert(shape, dtype, w, max_requests=8, max_steps=10, max_prefix=1 << 17):
    rosa = _rosa()
    cap = rosa.capacity(max_requests, 50, max_requests * 50, max_steps, max_prefix)
    return rosa.ActionExpert(shape, dtype, w, cap)


def _weights(shape, dtype):
    # the joint layout's weights fit the alternating one (same tensors)
    return cached_weights(dataclasses.replace(shape, attention_layout=0), dtype)


@pytest.mark.parametrize("shape,dtype,cases", [
    (TINY_ALT_SHAPE, "fp32", [(64, 8), (96, 8), (1, 3), (65, 5)]),
    (TINY_ALT_SHAPE, "bf16", [(64, 8), (96, 8), (1, 3), (65, 5)]),
    (PI0_ALT_SHAPE, "bf16", [(816, 50), (63, 16), (1, 1), (2048, 50), (65, 16)]),
])
@pytest.mark.parametrize("layer", [0, 1])
def test_attention_component_per_layer_kind(shape, dtype, cases, layer):
    e = _expert(shape, dtype, _weights(shape, dtype), max_prefix=1 << 16)
    qkv, qkv_d, o, structs, host, keep = _attn_case(e, cases, seed=11)
    e.attention(structs, layer, qkv_d, o)
    got = _thost(o)
    nq, nkv, hd = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    tol = 1e-5 if dtype == "fp32" else 1e-2
    M = sum(H for _, H in cases)
    assert np.isnan(got[M:]).all()
    for (P, H), (k, v, row, _) in zip(cases, host):
        rows = qkv[row:row + H].astype(np.float64)
        q = rows[:, : nq * hd].reshape(H, nq, hd)
        if layer % 2 == 0:          # cross-attention: the prefix only
            kf, vf = k[layer].astype(np.float64), v[layer].astype(np.float64)
        else:                       # self-attention: the action tokens only
            kf = rows[:, nq * hd:(nq + nkv) * hd].reshape(H, nkv, hd)
            vf = rows[:, (nq + nkv) * hd:].reshape(H, nkv, hd)
        ref = oracle_attention(q, kf, vf).reshape(H, nq * hd)
        err = rel_l2(got[row:row + H], ref)
        print(f"layer {layer} P={P} H={H}: rel-L2 {err:.2e}", flush=True)
        assert err < tol, (P, H, err)
    e.close()


def _run_check(shape, dtype, w, reqs, tol, label, expert=None):
    rosa = _rosa()
    e = expert or _expert(shape, dtype, w, max_requests=len(reqs))
    db = rosa.DeviceBatch(reqs, dtype)
    e.generate(db.structs)
    torch.cuda.synchronize()
    got = db.results()
    om = OracleModel(w, shape)
    for i, (g, r) in enumerate(zip(got, reqs)):
        err = rel_l2(g, om.generate([r])[0])
        print(f"{label} req {i} P={r.prefix_len} H={r.horizon} K={r.steps}: rel-L2 {err:.2e}", flush=True)
        assert err <= tol, (i, err)
    if expert is None:
        e.close()
    return got


def test_tiny_fp32_whole_call():
    w = _weights(TINY_ALT_SHAPE, "fp32")
    reqs = [custom_request(TINY_ALT_SHAPE, "fp32", P, H, K, seed=60 + i)
            for i, (P, H, K) in enumerate([(64, 8, 4), (1, 3, 2), (96, 5, 5), (33, 1, 1)])]
    _run_check(TINY_ALT_SHAPE, "fp32", w, reqs, 1e-5, "tiny fp32")


@pytest.mark.parametrize("isolate", [False, True])
def test_pi0_bf16_small_batch(isolate):
    w = _weights(PI0_ALT_SHAPE, "bf16")
    if isolate:   # MLP removed, attention gate biased to one: attention errors are visible
        w = {k: v.copy() for k, v in w.items()}
        d = PI0_ALT_SHAPE.d_model
        w["w_down"][:] = 0.0
        w["b_mod"][:, 2 * d:3 * d] = 1.0
    reqs = [custom_request(PI0_ALT_SHAPE, "bf16", P, H, K, seed=70 + i)
            for i, (P, H, K) in enumerate([(816, 50, 10), (1, 16, 5), (1500, 50, 5), (300, 1, 10), (65, 16, 10)])]
    _run_check(PI0_ALT_SHAPE, "bf16", w, reqs, 1e-2, "pi0-alt" + (" isolating" if isolate else ""))


def test_pi0_bf16_full_batch_two_lanes():
    # 160 factory requests: one item per query block, two lanes; sampled
    # requests against the oracle, and the one-lane result bitwise equal.
    rosa = _rosa()
    w = _weights(PI0_ALT_SHAPE, "bf16")
    preset = dataclasses.replace(PRESETS["factory_b256"], shape=PI0_ALT_SHAPE)
    reqs = make_requests(preset, indices=list(range(160)))
    e = _expert(PI0_ALT_SHAPE, "bf16", w, max_requests=160, max_prefix=160 * 1280)
    db = rosa.DeviceBatch(reqs, "bf16")
    outs = []
    for lanes in (2, 1):
        e.set_lanes(lanes)
        e.generate(db.structs)
        torch.cuda.synchronize()
        outs.append(db.results())
    for a, b in zip(outs[0], outs[1]):
        assert np.array_equal(a, b)
    om = OracleModel(w, PI0_ALT_SHAPE)
    for i in (0, 77, 159):
        err = rel_l2(outs[0][i], om.generate([reqs[i]])[0])
        print(f"full batch req {i}: rel-L2 {err:.2e}", flush=True)
        assert err <= 1e-2, (i, err)
    e.close()


def test_request_without_prefix_rejected():
    rosa = _rosa()
    w = _weights(TINY_ALT_SHAPE, "fp32")
    e = _expert(TINY_ALT_SHAPE, "fp32", w, max_requests=2)
    good = custom_request(TINY_ALT_SHAPE, "fp32", 8, 3, 2, seed=1)
    bad = custom_request(TINY_ALT_SHAPE, "fp32", 0, 3, 2, seed=2)
    db = rosa.DeviceBatch([good, bad], "fp32")
    assert e.generate_status(db.structs) == rosa.ROSA_E_INVALID
    torch.cuda.synchronize()
    assert np.isnan(db.results()[0]).all()        # nothing was enqueued
    e.close()
