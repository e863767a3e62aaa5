"""GPU parity of whole calls at the two head dimensions the other tests do not
run (64 and 128), against the float64 oracle: grouped-query attention with two
query heads per key head at head_dim 64, plain multi-head attention (one query
head per key head) at head_dim 128; both layouts (joint, alternating); fp32
and bf16.  Prefix lengths span several 32-key tiles, ragged tails and P = 0,
horizons a ragged query block and H = 1."""
import dataclasses

import numpy as np
import pytest

from oracle import OracleModel
from synthetic import custom_request
from tests.helpers import HD64_SHAPE as HD64, HD128_SHAPE as HD128, cached_weights, cap_for, rel_l2

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

# (P, H, K)
CASES = [(97, 17, 4), (0, 5, 3), (1, 1, 2), (64, 33, 5), (300, 50, 2)]


@pytest.mark.parametrize("layout", [0, 1])
@pytest.mark.parametrize("dtype,tol", [("fp32", 1e-5), ("bf16", 1e-2)])
@pytest.mark.parametrize("base", [HD64, HD128], ids=["hd64", "hd128"])
def test_whole_call_matches_oracle(base, dtype, tol, layout):
    from paper_2607_01088_amd import rosa
    shape = dataclasses.replace(base, attention_layout=layout)
    w = cached_weights(base, dtype)
    cases = [(max(P, 1) if layout == 1 else P, H, K) for P, H, K in CASES]   # alternating: P >= 1
    reqs = [custom_request(shape, dtype, P, H, K, seed=300 + i) for i, (P, H, K) in enumerate(cases)]
    e = rosa.ActionExpert(shape, dtype, w, cap_for(reqs))
    db = rosa.DeviceBatch(reqs, dtype)
    e.generate(db.structs)
    torch.cuda.synchronize()
    got = db.results()
    om = OracleModel(w, shape)
    for i, (g, r) in enumerate(zip(got, reqs)):
        want = om.generate([r])[0]
        err = rel_l2(g, want)
        print(f"hd={shape.head_dim} layout={layout} {dtype} req {i} P={r.prefix_len} H={r.horizon} "
              f"K={r.steps}: rel-L2 {err:.2e}", flush=True)
        disp = rel_l2(g - r.noise, want - r.noise)
        assert np.isfinite(g).all() and err <= tol, (i, err)
        if dtype == "bf16":
            assert disp <= tol, (i, disp)
    e.close()
