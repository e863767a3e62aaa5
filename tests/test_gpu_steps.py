"""Step-level batching (rosa_generate_steps and start_step): requests advanced
a few Euler steps per call, joining and leaving between calls, give the
results of the whole-chunk call (bitwise in fp32 mode, where no kernel's
arithmetic depends on the batch) and match the oracle; invalid resumption is
rejected."""
import numpy as np
import pytest

from oracle import OracleModel
from synthetic import PI0_SHAPE, TINY_SHAPE, custom_request
from tests.helpers import cached_weights, rel_l2

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _rosa():
    from paper_2607_01088_amd import rosa
    return rosa


class _Live:
    """One request on the device: prefix, noise, and the actions buffer that
    carries its Euler state between calls."""

    def __init__(self, r, dtype):
        rosa = _rosa()
        self.r = r
        self.k = rosa.to_device_kv(r.prefix_k, dtype) if r.prefix_len > 0 else None
        self.v = rosa.to_device_kv(r.prefix_v, dtype) if r.prefix_len > 0 else None
        self.noise = torch.from_numpy(np.ascontiguousarray(r.noise, dtype=np.float32)).cuda()
        self.out = torch.full_like(self.noise, float("nan"))
        self.done = 0

    def struct(self):
        return _rosa().request_struct(self.k, self.v, self.noise if self.done == 0 else None, self.out,
                                      self.r.prefix_len, self.r.horizon, self.r.steps, self.done)


def _schedule(expert, live, arrivals, per_call):
    """Each call: admit the requests whose arrival call has come, advance all
    in flight by at most per_call steps, retire the finished ones."""
    flight, t = [], 0
    while t < len(arrivals) or flight:
        flight += [live[i] for i, a in enumerate(arrivals) if a == t]
        if flight:
            expert.generate_steps([x.struct() for x in flight], per_call)
            torch.cuda.synchronize()
            for x in flight:
                x.done = min(x.r.steps, x.done + per_call)
            flight = [x for x in flight if x.done < x.r.steps]
        t += 1
        assert t < 1000
    return [x.out.cpu().numpy() for x in live]


def _requests(shape, dtype, n, seed, max_p=80):
    rng = np.random.default_rng(seed)
    return [custom_request(shape, dtype, int(rng.integers(0, max_p)), int(rng.choice([1, 3, 8])),
                           int(rng.choice([1, 2, 4, 5])), seed * 100 + i) for i in range(n)]


@pytest.mark.parametrize("per_call", [1, 2, 3])
def test_fp32_pieces_equal_whole_calls_bitwise(per_call):
    rosa = _rosa()
    w = cached_weights(TINY_SHAPE, "fp32")
    reqs = _requests(TINY_SHAPE, "fp32", 7, 5)
    cap = rosa.capacity(8, 8, 64, 5, 1 << 10)
    e = rosa.ActionExpert(TINY_SHAPE, "fp32", w, cap)
    db = rosa.DeviceBatch(reqs, "fp32")
    e.generate(db.structs)
    torch.cuda.synchronize()
    whole = db.results()
    live = [_Live(r, "fp32") for r in reqs]
    got = _schedule(e, live, [0, 0, 1, 1, 2, 4, 6], per_call)
    for i, (g, ref) in enumerate(zip(got, whole)):
        assert np.array_equal(g, ref), i
    om = OracleModel(w, TINY_SHAPE)
    for g, r in zip(got, reqs):
        assert rel_l2(g, om.generate([r])[0]) <= 1e-5
    e.close()


def test_bf16_continuous_schedule_matches_oracle():
    rosa = _rosa()
    w = cached_weights(PI0_SHAPE, "bf16")
    reqs = _requests(PI0_SHAPE, "bf16", 6, 9, max_p=300)
    cap = rosa.capacity(8, 8, 64, 5, 8 * 300)
    e = rosa.ActionExpert(PI0_SHAPE, "bf16", w, cap)
    live = [_Live(r, "bf16") for r in reqs]
    got = _schedule(e, live, [0, 0, 0, 1, 2, 3], 1)
    om = OracleModel(w, PI0_SHAPE)
    for i, (g, r) in enumerate(zip(got, reqs)):
        err = rel_l2(g, om.generate([r])[0])
        print(f"req {i} P={r.prefix_len} H={r.horizon} K={r.steps}: rel-L2 {err:.3e}", flush=True)
        assert err <= 1e-2, (i, err)
    e.close()


def test_resumption_is_validated():
    rosa = _rosa()
    w = cached_weights(TINY_SHAPE, "fp32")
    r = custom_request(TINY_SHAPE, "fp32", 8, 3, 4, 1)
    cap = rosa.capacity(2, 8, 16, 4, 64)
    e = rosa.ActionExpert(TINY_SHAPE, "fp32", w, cap)
    x = _Live(r, "fp32")
    x.done = 4                                   # start_step == K: nothing left
    assert e.generate_status([x.struct()]) == rosa.ROSA_E_INVALID
    x.done = 0
    with pytest.raises(rosa.RosaError):
        e.generate_steps([x.struct()], 0)       # max_steps < 1
    e.close()
