"""Host-side checks of the C ABI: the library loads and exports every declared
function, validation is all-or-nothing with the documented status codes, and
the batch plan (K-descending order, token offsets, active tokens per step,
distinct flow times) is right.  No GPU needed."""
import ctypes as C

import pytest

from paper_2607_01088_amd import rosa
from synthetic import PI0_SHAPE, TINY_SHAPE
from tests.helpers import declared_functions

FAKE = 0x1000   # non-NULL device address; host planning never dereferences it


def req(P, H, K, k=FAKE, v=FAKE, noise=FAKE, out=FAKE, start_step=0):
    return rosa.request_struct(k, v, noise, out, P, H, K, start_step)


def test_library_exports_every_declared_function():
    lib = rosa.load()
    names = declared_functions()
    assert "rosa_batch_create" in names and "rosa_generate_actions" in names and "rosa_destroy" in names
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    lib = rosa.load()
    for s in range(6):
        assert lib.rosa_status_string(s)
    assert lib.rosa_status_string(99) == b"unknown status"


def test_create_rejects_null_and_bad_shapes_before_touching_the_gpu():
    lib = rosa.load()
    h = C.c_void_p()
    assert lib.rosa_batch_create(None, None, None, None, C.byref(h)) == rosa.ROSA_E_INVALID
    assert not h.value
    cfg = rosa.model_config(TINY_SHAPE, "fp32")
    cap = rosa.capacity(2, 8, 16, 4, 200)
    w = rosa.Weights()
    assert lib.rosa_batch_create(C.byref(cfg), C.byref(w), C.byref(cap), None, C.byref(h)) == rosa.ROSA_E_INVALID
    cfg.head_dim = 48
    assert lib.rosa_batch_create(C.byref(cfg), C.byref(w), C.byref(cap), None, C.byref(h)) \
        == rosa.ROSA_E_UNSUPPORTED
    assert lib.rosa_last_error(None)
    assert lib.rosa_generate_actions(None, None, 0) == rosa.ROSA_E_INVALID
    lib.rosa_destroy(None)   # NULL-safe


def _plan(reqs, cap=None, shape=PI0_SHAPE, dtype="bf16"):
    cap = cap or rosa.capacity(16, 50, 400, 10, 100000)
    return rosa.plan(shape, dtype, cap, reqs)


def test_plan_sorts_by_steps_and_prefixes_active_tokens():
    reqs = [req(1000, 16, 5), req(2000, 50, 10), req(0, 16, 10), req(700, 50, 5)]
    st, order, tok, mk, counts = _plan(reqs)
    assert st == rosa.ROSA_OK
    assert order == [1, 2, 0, 3]                         # K descending, stable
    assert tok == [66, 0, 50, 82]                        # offsets follow the plan order
    assert mk == [132] * 5 + [66] * 5
    n_tau, n_items, n_qb, n_split = counts
    assert n_tau == 10                                   # {k/5} is a subset of {k/10}
    assert n_qb == 1 + 4 + 1 + 4                         # ceil(8H/128) per request
    # a small batch splits long key ranges (>= 64 keys per item); short ones stay whole
    assert n_items > n_qb and n_split > 0


def test_plan_distinct_taus_counts_fp32_division():
    reqs = [req(1, 2, 3), req(1, 2, 4), req(1, 2, 6)]
    st, _, _, _, counts = _plan(reqs)
    assert st == rosa.ROSA_OK
    taus = {k / K for K in (3, 4, 6) for k in range(K)}
    import numpy as np
    taus32 = {float(np.float32(k) / np.float32(K)) for K in (3, 4, 6) for k in range(K)}
    assert counts[0] == len(taus32) == len(taus)


def test_plan_no_split_for_a_full_batch():
    reqs = [req(600, 50, 10) for _ in range(160)]       # 640 query blocks >= split target
    cap = rosa.capacity(256, 50, 256 * 50, 10, 256 * 2048)
    st, _, _, _, counts = _plan(reqs, cap)
    assert st == rosa.ROSA_OK
    assert counts[1] == counts[2] == 640 and counts[3] == 0


def test_plan_lanes_balance_and_cover_every_request():
    """Lane assignment (rosa_debug_plan_lanes): every request gets a lane, both
    lanes of a 256-request factory-shaped set carry similar work, and fewer
    than 64 requests per lane keep a single lane."""
    import numpy as np
    rng = np.random.default_rng(1)
    reqs = [req(int(rng.integers(512, 1281)), int(rng.choice([16, 50])), int(rng.choice([5, 10]))) for _ in range(256)]
    cap = rosa.capacity(256, 50, 256 * 50, 10, 256 * 1280)
    st, lanes = rosa.plan_lanes(PI0_SHAPE, "bf16", cap, reqs, 2)
    assert st == rosa.ROSA_OK and sorted(set(lanes)) == [0, 1]
    work = [0.0, 0.0]
    for r, l in zip(reqs, lanes):
        work[l] += r.horizon * r.num_steps * (1.0 + (r.prefix_len + r.horizon) / 1800.0)
    assert abs(work[0] - work[1]) / sum(work) < 0.01
    st, lanes = rosa.plan_lanes(PI0_SHAPE, "bf16", cap, reqs[:100], 2)
    assert st == rosa.ROSA_OK and set(lanes) == {0}
    st, lanes = rosa.plan_lanes(PI0_SHAPE, "fp32", cap, reqs, 2)
    assert st == rosa.ROSA_OK and set(lanes) == {0}


def _walk_lists(nb, item_of, nxt):
    """Follow each block's chain; returns the item lists per block."""
    seen = [False] * len(item_of)
    blocks = []
    for b in range(nb):
        lst, e = [], b
        while e >= 0:
            assert 0 <= e < len(item_of) and not seen[e], (b, e)
            seen[e] = True
            if item_of[e] < 0:
                assert e == b and nxt[e] == -1      # idle: a first entry with no successor
                break
            lst.append(item_of[e])
            e = nxt[e]
        blocks.append(lst)
    assert all(seen), "every table entry belongs to one block's chain"
    return blocks


@pytest.mark.parametrize("case", ["factory", "one_request", "few_requests"])
def test_attention_launch_lists_cover_every_item_once_and_balance(case):
    """Persistent attention launch lists (rosa_debug_attn_lists): every work
    item of the launch is on exactly one block's chain, the grid is a multiple
    of the 8 XCDs and at most 512 blocks, block loads are within one item of
    the mean (longest-processing-time bound), and while there are no more
    items than blocks no block runs two."""
    import numpy as np
    rng = np.random.default_rng(5)
    if case == "factory":
        reqs = [req(int(rng.integers(512, 1281)), int(rng.choice([16, 50])), int(rng.choice([5, 10])))
                for _ in range(256)]
    elif case == "one_request":
        reqs = [req(1024, 50, 10)]
    else:
        reqs = [req(int(rng.integers(600, 1025)), 50, 10) for _ in range(5)]
    cap = rosa.capacity(len(reqs), 50, len(reqs) * 50, 10, len(reqs) * 1280)
    st, _, _, _, counts = rosa.plan(PI0_SHAPE, "bf16", cap, reqs)
    assert st == rosa.ROSA_OK
    n_items = counts[1]
    st, nb, item_of, nxt, cost = rosa.attn_lists(PI0_SHAPE, cap, reqs, n_items)
    assert st == rosa.ROSA_OK
    assert nb % 8 == 0 and 8 <= nb <= 512
    blocks = _walk_lists(nb, item_of, nxt)
    flat = sorted(i for lst in blocks for i in lst)
    assert flat == list(range(n_items))
    over = 6                                  # fixed per-item overhead the packing charges, in steps
    loads = [sum(cost[i] + over for i in lst) for lst in blocks]
    biggest = max(cost) + over
    assert max(loads) <= sum(loads) / nb + biggest
    if n_items <= nb:
        assert max(len(lst) for lst in blocks) == 1
    st, *_ = rosa.attn_lists(PI0_SHAPE, cap, reqs[:0], 0)
    assert st == rosa.ROSA_OK


@pytest.mark.parametrize("bad,status", [
    (dict(P=-1), rosa.ROSA_E_INVALID),
    (dict(H=0), rosa.ROSA_E_INVALID),
    (dict(H=51), rosa.ROSA_E_INVALID),
    (dict(K=0), rosa.ROSA_E_INVALID),
    (dict(K=11), rosa.ROSA_E_INVALID),
    (dict(noise=None), rosa.ROSA_E_INVALID),
    (dict(out=None), rosa.ROSA_E_INVALID),
    (dict(k=None), rosa.ROSA_E_INVALID),
    (dict(start_step=5), rosa.ROSA_E_INVALID),
    (dict(start_step=-1), rosa.ROSA_E_INVALID),
])
def test_plan_validation_all_or_nothing(bad, status):
    args = dict(P=10, H=16, K=5, k=FAKE, v=FAKE, noise=FAKE, out=FAKE, start_step=0)
    args.update(bad)
    good = req(5, 8, 5)
    bad_req = req(args["P"], args["H"], args["K"], args["k"], args["v"], args["noise"], args["out"], args["start_step"])
    st, *_ = _plan([good, bad_req, good])
    assert st == status


def test_plan_resumed_request_needs_no_noise():
    # a request resumed at step 2 of 5 reads its state from actions and runs
    # its remaining 3 steps; the fresh one runs all 4 and comes first
    st, order, tok, m_k, counts = _plan([req(10, 16, 5, noise=None, start_step=2), req(5, 8, 4)])
    assert st == rosa.ROSA_OK
    assert order == [1, 0]
    assert m_k[:5] == [24, 24, 24, 8, 0]


def test_plan_null_prefix_allowed_when_empty():
    st, *_ = _plan([req(0, 8, 2, k=None, v=None)])
    assert st == rosa.ROSA_OK


def test_plan_capacity_limits():
    cap = rosa.capacity(2, 50, 60, 10, 1000)
    assert _plan([req(10, 8, 2)] * 3, cap)[0] == rosa.ROSA_E_CAPACITY          # too many requests
    assert _plan([req(10, 50, 2), req(10, 16, 2)], cap)[0] == rosa.ROSA_E_CAPACITY  # sum H
    assert _plan([req(600, 8, 2), req(600, 8, 2)], cap)[0] == rosa.ROSA_E_CAPACITY  # sum P
    assert _plan([], cap)[0] == rosa.ROSA_OK


def test_plan_too_many_distinct_taus():
    cap = rosa.capacity(64, 8, 512, 64, 1000)
    reqs = [req(1, 1, K) for K in range(40, 64)]
    assert _plan(reqs, cap, shape=TINY_SHAPE)[0] == rosa.ROSA_E_CAPACITY


def test_plan_alternating_layout():
    # Two attention sets: cross-attention items over the prefix and
    # self-attention items over the actions, each one item per query block at
    # this batch size; a request without a prefix is rejected.
    from synthetic import PI0_ALT_SHAPE
    reqs = [req(600, 50, 10) for _ in range(160)]
    cap = rosa.capacity(256, 50, 256 * 50, 10, 256 * 2048)
    st, _, _, _, counts = _plan(reqs, cap, shape=PI0_ALT_SHAPE)
    assert st == rosa.ROSA_OK
    assert counts[2] == 640 and counts[1] == 2 * 640 and counts[3] == 0
    st, *_ = _plan([req(5, 8, 5), req(0, 8, 5, k=None, v=None)], shape=PI0_ALT_SHAPE)
    assert st == rosa.ROSA_E_INVALID
    # small batch: the prefix keys split over items (partial slots), the
    # 50 self-attention keys (fewer than the 64 a split item needs) do not
    st, _, _, _, counts = _plan([req(1200, 50, 10)], shape=PI0_ALT_SHAPE)
    assert st == rosa.ROSA_OK
    assert counts[3] == counts[2] and counts[1] > 2 * counts[2]


def test_create_rejects_unknown_layout():
    lib = rosa.load()
    h = C.c_void_p()
    cfg = rosa.model_config(TINY_SHAPE, "fp32")
    cfg.attention_layout = 2
    cap = rosa.capacity(2, 8, 16, 4, 200)
    w = rosa.Weights()      # NULL weights would be rejected later, with another message
    assert lib.rosa_batch_create(C.byref(cfg), C.byref(w), C.byref(cap), None, C.byref(h)) == rosa.ROSA_E_INVALID
    assert not h.value
    assert b"configuration" in lib.rosa_last_error(None)


def test_prefill_create_validates_before_touching_the_gpu():
    from synthetic import TINY_VLM
    lib = rosa.load()
    h = C.c_void_p()
    w = rosa.VlmWeights()
    buf = (C.c_float * 4)()
    for f in ("w_qkv", "w_o", "w_up", "w_down"):
        setattr(w, f, C.cast(buf, C.POINTER(C.c_float)))
    cases = [rosa.vlm_config(TINY_VLM, "fp32", head_layers=2),      # context form without w_ctx
             rosa.vlm_config(TINY_VLM, "fp32")]
    cases[1].cache_form = 5
    bad_layers = rosa.vlm_config(TINY_VLM, "fp32", head_layers=2)
    bad_layers.head_layers = 0
    cases.append(bad_layers)
    for base in (0.5, 1.0, -1.0, float("inf"), float("nan")):   # rotary base: 0 (none) or > 1
        bad_rope = rosa.vlm_config(TINY_VLM, "fp32")
        bad_rope.rope_base = base
        cases.append(bad_rope)
    for cfg in cases:
        assert lib.rosa_prefill_create(C.byref(cfg), C.byref(w), 1, 8, None, C.byref(h)) == rosa.ROSA_E_INVALID
        assert not h.value and lib.rosa_prefill_last_error(None)
    cfg = rosa.vlm_config(TINY_VLM, "fp32")
    cfg.head_dim = 48
    assert lib.rosa_prefill_create(C.byref(cfg), C.byref(w), 1, 8, None, C.byref(h)) == rosa.ROSA_E_UNSUPPORTED
    assert lib.rosa_prefill_run(None, None, 0) == rosa.ROSA_E_INVALID
    lib.rosa_prefill_destroy(None)


def test_create_rejects_query_row_counts_above_int32_range():
    # a request's or job's query rows (tokens x query heads per KV head) are int32
    from synthetic import TINY_VLM
    lib = rosa.load()
    h = C.c_void_p()
    cfg = rosa.model_config(TINY_SHAPE, "fp32")                 # 4 query heads per KV head
    cap = rosa.capacity(2, 1 << 29, 1 << 29, 4, 200)
    w = rosa.Weights()
    assert lib.rosa_batch_create(C.byref(cfg), C.byref(w), C.byref(cap), None, C.byref(h)) \
        == rosa.ROSA_E_UNSUPPORTED
    vcfg = rosa.vlm_config(TINY_VLM, "fp32")
    assert lib.rosa_prefill_create(C.byref(vcfg), C.byref(rosa.VlmWeights()), 1, 1 << 29, None, C.byref(h)) \
        == rosa.ROSA_E_UNSUPPORTED
    assert not h.value
