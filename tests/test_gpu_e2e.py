"""End-to-end GPU parity of rosa_generate_actions against the CPU oracle, plus
the bit-exact indexing checks (zero and constant velocity), batch invariance,
a mutation check that the gate can see attention, and ABI error handling."""
import dataclasses

import numpy as np
import pytest

from oracle import OracleModel
from synthetic import (PI0_SHAPE, PRESETS, TINY_SHAPE, custom_request, make_metadata, make_requests,
                       make_weights)
from tests.helpers import cached_weights, rel_l2

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _rosa():
    from paper_2607_01088_amd import rosa
    return rosa


def _expert(shape, dtype, weights, max_requests=16, max_tokens=None, max_steps=10, max_prefix=1 << 17):
    rosa = _rosa()
    cap = rosa.capacity(max_requests, 50, max_tokens or max_requests * 50, max_steps, max_prefix)
    return rosa.ActionExpert(shape, dtype, weights, cap)


def _run(expert, requests, dtype):
    db = _rosa().DeviceBatch(requests, dtype)
    expert.generate(db.structs)
    torch.cuda.synchronize()
    return db.results(), db


def _check(got, requests, weights, shape, tol, label):
    """Each chunk against the oracle: rel-L2 of x_K, and (bf16 gate) rel-L2 of
    the displacement x_K - x_0, which attention moves by a larger fraction
    than it moves x_K."""
    om = OracleModel(weights, shape)
    worst = 0.0
    for i, (g, r) in enumerate(zip(got, requests)):
        ref = om.generate([r])[0]
        err = rel_l2(g, ref)
        disp = rel_l2(g - r.noise, ref - r.noise)
        print(f"{label} req {i} P={r.prefix_len} H={r.horizon} K={r.steps}: rel-L2 {err:.3e} "
              f"(displacement {disp:.3e})", flush=True)
        worst = max(worst, err)
        assert err <= tol, (i, err)
        if tol >= 1e-3:
            assert disp <= tol, (i, disp)
    return worst


@pytest.fixture(scope="module")
def pi0_expert():
    w = cached_weights(PI0_SHAPE, "bf16")
    e = _expert(PI0_SHAPE, "bf16", w, max_requests=256, max_prefix=256 * 1280)
    yield e, w
    e.close()


# ------------------------------------------------------------------ presets vs oracle

def test_tiny_fp32_preset():
    p = PRESETS["tiny"]
    w = make_weights(p.shape, "fp32")
    reqs = make_requests(p)
    e = _expert(p.shape, "fp32", w)
    got, _ = _run(e, reqs, "fp32")
    _check(got, reqs, w, p.shape, 1e-5, "tiny fp32")
    e.close()


def test_tiny_bf16_preset():
    p = dataclasses.replace(PRESETS["tiny"], dtype="bf16")
    w = make_weights(p.shape, "bf16")
    reqs = make_requests(p)
    e = _expert(p.shape, "bf16", w)
    got, _ = _run(e, reqs, "bf16")
    _check(got, reqs, w, p.shape, 1e-2, "tiny bf16")
    e.close()


def test_pi0_b1_preset(pi0_expert):
    e, w = pi0_expert
    reqs = make_requests(PRESETS["pi0_b1"])
    got, _ = _run(e, reqs, "bf16")
    _check(got, reqs, w, PI0_SHAPE, 1e-2, "pi0_b1")


def test_factory_subset_mixed_horizons_and_steps(pi0_expert):
    e, w = pi0_expert
    p = PRESETS["factory_b256"]
    meta = make_metadata(p)
    idx = []
    for H in (16, 50):
        for K in (5, 10):
            idx += [i for i, m in enumerate(meta) if m.horizon == H and m.steps == K][:2]
    reqs = make_requests(p, indices=idx)
    got, _ = _run(e, reqs, "bf16")
    _check(got, reqs, w, PI0_SHAPE, 1e-2, "factory subset")


@pytest.mark.timeout(900)
def test_factory_b256_full_batch_sampled(pi0_expert):
    """The benchmark's workload, whole batch in one call; sampled requests
    (one per horizon/step class, plus the longest and shortest prefix) checked
    one by one against the oracle."""
    e, w = pi0_expert
    p = PRESETS["factory_b256"]
    reqs = make_requests(p)
    got, _ = _run(e, reqs, "bf16")
    meta = make_metadata(p)
    pick = set()
    for H in (16, 50):
        for K in (5, 10):
            pick.add(next(i for i, m in enumerate(meta) if m.horizon == H and m.steps == K))
    pick.add(int(np.argmax([m.prefix_len for m in meta])))
    pick.add(int(np.argmin([m.prefix_len for m in meta])))
    pick = sorted(pick)
    for g in got:
        assert np.isfinite(g).all()
    _check([got[i] for i in pick], [reqs[i] for i in pick], w, PI0_SHAPE, 1e-2, "factory_b256")


@pytest.mark.timeout(900)
def test_pi0_b32_preset_sampled(pi0_expert):
    """The 32-robot pi0 preset (prefixes 600-1024 tokens, each with its own KV
    cache) in one call: the longest and shortest prefix and two more requests
    against the oracle, every chunk finite."""
    e, w = pi0_expert
    p = PRESETS["pi0_b32"]
    reqs = make_requests(p)
    got, _ = _run(e, reqs, "bf16")
    meta = make_metadata(p)
    pick = sorted({int(np.argmax([m.prefix_len for m in meta])), int(np.argmin([m.prefix_len for m in meta])), 7, 20})
    for g in got:
        assert np.isfinite(g).all()
    _check([got[i] for i in pick], [reqs[i] for i in pick], w, PI0_SHAPE, 1e-2, "pi0_b32")


def test_factory_first16_deferred_norms(pi0_expert):
    """Sixteen robots (528 rows): every output projection and MLP-down either
    folds the next norm into its K-slice reduction or defers it to the next
    product, so the only norm launches left are each step's first; four
    requests (one per horizon x steps class) against the oracle."""
    e, w = pi0_expert
    p = PRESETS["factory_b256"]
    reqs = make_requests(p, indices=list(range(16)))
    meta = make_metadata(p)[:16]
    db = _rosa().DeviceBatch(reqs, "bf16")
    e.set_profiling(True)
    try:
        e.generate(db.structs)
        torch.cuda.synchronize()
        prof = e.profile()
    finally:
        e.set_profiling(False)
    k_max = max(m.steps for m in meta)
    assert prof["modnorm"][0] == k_max, prof["modnorm"]
    # the time MLP's four launches and the shift table of the deferred norms
    assert prof["time_conditioning"][0] == 5, prof["time_conditioning"]
    got = db.results()
    pick = []
    for cls in sorted({(m.horizon, m.steps) for m in meta}):
        pick.append(next(i for i, m in enumerate(meta) if (m.horizon, m.steps) == cls))
    _check([got[i] for i in pick], [reqs[i] for i in pick], w, PI0_SHAPE, 1e-2, "factory first 16")


@pytest.mark.timeout(900)
def test_factory_b256_attention_isolating_both_lanes():
    """The benchmark's whole batch with the MLP removed and the attention gate
    biased to one, so that attention decides the result: the default call
    (two lanes, per-step launch lists), checked on one request per
    horizon x steps class in each lane plus the longest and shortest prefix
    among each lane's ten-step requests (the only ones active in steps 5-9)."""
    from paper_2607_01088_amd import rosa
    base = cached_weights(PI0_SHAPE, "bf16")
    w = _attention_isolating(base, PI0_SHAPE)
    p = PRESETS["factory_b256"]
    meta = make_metadata(p)
    e = _expert(PI0_SHAPE, "bf16", w, max_requests=256, max_prefix=256 * 1280)
    reqs = make_requests(p)
    db = rosa.DeviceBatch(reqs, "bf16")
    st, lanes = rosa.plan_lanes(PI0_SHAPE, "bf16", e.cap, db.structs, 2)
    assert st == 0 and sorted(set(lanes)) == [0, 1]
    e.generate(db.structs)
    torch.cuda.synchronize()
    got = db.results()
    for g in got:
        assert np.isfinite(g).all()
    pick = set()
    for lane in (0, 1):
        mine = [i for i in range(len(meta)) if lanes[i] == lane]
        for H in (16, 50):
            for K in (5, 10):
                pick.add(next(i for i in mine if meta[i].horizon == H and meta[i].steps == K))
        ten = [i for i in mine if meta[i].steps == 10]
        pick.add(max(ten, key=lambda i: meta[i].prefix_len))
        pick.add(min(ten, key=lambda i: meta[i].prefix_len))
    pick = sorted(pick)
    print("lanes of the checked requests:", [lanes[i] for i in pick], flush=True)
    _check([got[i] for i in pick], [reqs[i] for i in pick], w, PI0_SHAPE, 1e-2, "factory_b256 isolating")
    e.close()


@pytest.mark.timeout(900)
def test_stress_b512_full_batch_sampled():
    """The largest preset: 512 requests with 1024-2048-token prefixes (14.5 GB
    of prefix KV resident) in one call; the longest and shortest prefix and
    one more request against the oracle, every result finite."""
    w = cached_weights(PI0_SHAPE, "bf16")
    p = PRESETS["stress_b512"]
    meta = make_metadata(p)
    e = _expert(PI0_SHAPE, "bf16", w, max_requests=512, max_prefix=sum(m.prefix_len for m in meta))
    reqs = make_requests(p, threads=16)
    got, db = _run(e, reqs, "bf16")
    del db
    pick = sorted({int(np.argmax([m.prefix_len for m in meta])), int(np.argmin([m.prefix_len for m in meta])), 300})
    for g in got:
        assert np.isfinite(g).all()
    _check([got[i] for i in pick], [reqs[i] for i in pick], w, PI0_SHAPE, 1e-2, "stress_b512")
    e.close()


# ------------------------------------------------------------------ attention must be visible

def _attention_isolating(w, shape):
    w = {k: v.copy() for k, v in w.items()}
    d = shape.d_model
    w["w_down"][:] = 0.0
    w["b_mod"][:, 2 * d:3 * d] = 1.0
    return w


def test_attention_isolating_variant_and_prefix_swap():
    """MLP removed, attention gate biased to 1: parity holds, and swapping two
    requests' prefix caches moves the result far outside the tolerance."""
    base = cached_weights(PI0_SHAPE, "bf16")
    w = _attention_isolating(base, PI0_SHAPE)
    e = _expert(PI0_SHAPE, "bf16", w, max_requests=2)
    reqs = [custom_request(PI0_SHAPE, "bf16", 816, 50, 10, seed=40),
            custom_request(PI0_SHAPE, "bf16", 700, 16, 5, seed=41)]
    got, db = _run(e, reqs, "bf16")
    _check(got, reqs, w, PI0_SHAPE, 1e-2, "attention-isolating")
    rosa = _rosa()
    s0, s1 = db.structs
    swapped = [rosa.request_struct(db.k[1], db.v[1], db.noise[0], db.actions[0], 700, 50, 10),
               rosa.request_struct(db.k[0], db.v[0], db.noise[1], db.actions[1], 816, 16, 5)]
    e.generate(swapped)
    torch.cuda.synchronize()
    moved = rel_l2(db.actions[0].cpu().numpy(), got[0])
    print(f"prefix swap moves request 0 by rel-L2 {moved:.3e}", flush=True)
    assert moved > 5e-2
    e.close()


# ------------------------------------------------------------------ bit-exact indexing

def _grid_noise(rng, H, A):
    return (np.round(rng.uniform(-4, 4, size=(H, A)) * 256) / 256).astype(np.float32)


@pytest.mark.parametrize("shape,dtype", [(TINY_SHAPE, "fp32"), (TINY_SHAPE, "bf16"), (PI0_SHAPE, "bf16")])
def test_zero_velocity_returns_noise_bitwise(shape, dtype):
    w = dict(cached_weights(shape, dtype))
    w["w_out"] = np.zeros_like(w["w_out"])
    w["b_out"] = np.zeros_like(w["b_out"])
    e = _expert(shape, dtype, w, max_requests=8)
    reqs = [custom_request(shape, dtype, P, H, K, seed=50 + i)
            for i, (P, H, K) in enumerate([(64, 16, 5), (0, 50, 10), (300, 1, 3), (96, 50, 1), (1, 16, 10)])]
    got, _ = _run(e, reqs, dtype)
    for g, r in zip(got, reqs):
        assert np.array_equal(g, r.noise)
    e.close()


@pytest.mark.parametrize("shape,dtype", [(TINY_SHAPE, "fp32"), (TINY_SHAPE, "bf16"), (PI0_SHAPE, "bf16")])
def test_constant_velocity_closed_form(shape, dtype):
    w = {k: np.zeros_like(v) for k, v in cached_weights(shape, dtype).items()}
    rng = np.random.default_rng(9)
    c = (np.round(rng.uniform(-2, 2, size=shape.action_dim) * 16) / 16).astype(np.float32)
    w["b_out"] = c
    e = _expert(shape, dtype, w, max_requests=8)
    specs = [(40, 16, 1), (0, 50, 2), (7, 5, 4), (120, 16, 8), (33, 50, 5), (64, 3, 10)]
    reqs = []
    for i, (P, H, K) in enumerate(specs):
        r = custom_request(shape, dtype, P, H, K, seed=60 + i)
        r.noise = _grid_noise(rng, H, shape.action_dim)
        reqs.append(r)
    got, _ = _run(e, reqs, dtype)
    for g, r in zip(got, reqs):
        expect = r.noise + c
        if r.steps in (1, 2, 4, 8):
            assert np.array_equal(g, expect), r.steps
        else:
            assert np.max(np.abs(g - expect)) <= 1e-6 * np.max(np.abs(expect)) * 8, r.steps
    e.close()


# ------------------------------------------------------------------ invariances

def test_batch_and_permutation_invariance(pi0_expert):
    e, w = pi0_expert
    p = PRESETS["factory_b256"]
    reqs = make_requests(p, indices=list(range(6)))
    batched, _ = _run(e, reqs, "bf16")
    perm = [3, 0, 5, 1, 4, 2]
    permuted, _ = _run(e, [reqs[i] for i in perm], "bf16")
    for j, i in enumerate(perm):
        assert rel_l2(permuted[j], batched[i]) <= 1e-3
    for i, r in enumerate(reqs):
        alone, _ = _run(e, [r], "bf16")
        err = rel_l2(alone[0], batched[i])
        print(f"request {i}: alone vs batched rel-L2 {err:.3e}", flush=True)
        assert err <= 1e-3


def test_repeat_runs_are_bitwise_identical(pi0_expert):
    e, _ = pi0_expert
    reqs = make_requests(PRESETS["factory_b256"], indices=list(range(10, 18)))
    db = _rosa().DeviceBatch(reqs, "bf16")
    outs = []
    for _ in range(5):
        e.generate(db.structs)
        torch.cuda.synchronize()
        outs.append(db.results())
    for o in outs[1:]:
        for a, b in zip(o, outs[0]):
            assert np.array_equal(a, b)


def test_projection_block_configs_bitwise_identical(pi0_expert):
    """The whole call gives bitwise the same actions whichever projection
    block configuration is forced.  The default path may split K over blocks
    for launches with few tiles (this 4-request batch), which sums in another
    order: the same actions to rounding."""
    e, _ = pi0_expert
    reqs = make_requests(PRESETS["factory_b256"], indices=[0, 7, 21, 40])
    db = _rosa().DeviceBatch(reqs, "bf16")
    outs = []
    n_cfg = e.gemm_config(-1)
    try:
        for cfg in [-1] + list(range(n_cfg)):
            e.gemm_config(cfg)
            e.generate(db.structs)
            torch.cuda.synchronize()
            outs.append(db.results())
    finally:
        e.gemm_config(-1)
    for o in outs[2:]:
        for a, b in zip(o, outs[1]):
            assert np.array_equal(a, b)
    for a, b in zip(outs[0], outs[1]):
        assert rel_l2(a, b) < 5e-3


def test_lane_counts_bitwise_identical(pi0_expert):
    """Splitting the call into concurrent sub-batches (lanes) does not change
    any request's actions."""
    e, _ = pi0_expert
    reqs = make_requests(PRESETS["factory_b256"], indices=list(range(128)))
    db = _rosa().DeviceBatch(reqs, "bf16")
    outs = []
    try:
        for lanes in (1, 2):
            e.set_lanes(lanes)
            e.generate(db.structs)
            torch.cuda.synchronize()
            outs.append(db.results())
    finally:
        e.set_lanes(2)
    for o in outs[1:]:
        for a, b in zip(o, outs[0]):
            assert np.array_equal(a, b)


# ------------------------------------------------------------------ ABI errors on a live handle

def test_invalid_request_enqueues_nothing(pi0_expert):
    rosa = _rosa()
    e, _ = pi0_expert
    reqs = make_requests(PRESETS["pi0_b1"])
    db = rosa.DeviceBatch(reqs, "bf16")
    good = db.structs[0]
    bad = rosa.request_struct(db.k[0], db.v[0], db.noise[0], db.actions[0], 816, 51, 10)
    st = e.generate_status([good, bad])
    assert st == rosa.ROSA_E_INVALID
    torch.cuda.synchronize()
    assert torch.isnan(db.actions[0]).all()           # sentinel untouched: nothing ran
    assert e.generate_status([]) == rosa.ROSA_OK
    e.generate([good])                                 # the handle still works
    torch.cuda.synchronize()
    assert torch.isfinite(db.actions[0]).all()
