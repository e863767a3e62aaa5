"""Two handles used at the same time on two streams (default priority) share
no state: each gives bitwise the results it gives alone, and a prefix
producer and an expert can run concurrently on their own streams."""
import numpy as np
import pytest

from synthetic import PRESETS, TINY_SHAPE, TINY_VLM, make_prefix_embeddings, make_requests, make_vlm_weights
from tests.helpers import cached_weights

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def test_two_experts_on_two_streams():
    from paper_2607_01088_amd import rosa
    p = PRESETS["factory_b256"]
    w = cached_weights(p.shape, "bf16")
    ra = make_requests(p, indices=list(range(0, 6)))
    rb = make_requests(p, indices=list(range(40, 44)))
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    cap = rosa.capacity(8, 50, 400, 10, 8 * 1280)
    ea = rosa.ActionExpert(p.shape, "bf16", w, cap, stream=sa.cuda_stream)
    eb = rosa.ActionExpert(p.shape, "bf16", w, cap, stream=sb.cuda_stream)
    da, db = rosa.DeviceBatch(ra, "bf16"), rosa.DeviceBatch(rb, "bf16")
    torch.cuda.synchronize()
    ea.generate(da.structs)
    torch.cuda.synchronize()
    alone_a = da.results()
    eb.generate(db.structs)
    torch.cuda.synchronize()
    alone_b = db.results()
    for _ in range(3):
        ea.generate(da.structs)
        eb.generate(db.structs)
    torch.cuda.synchronize()
    for x, y in zip(da.results(), alone_a):
        assert np.array_equal(x, y)
    for x, y in zip(db.results(), alone_b):
        assert np.array_equal(x, y)
    ea.close()
    eb.close()


def test_prefill_and_expert_on_two_streams():
    from paper_2607_01088_amd import rosa
    w = make_vlm_weights(TINY_VLM, "fp32")
    lens = [40, 77]
    emb = [torch.from_numpy(make_prefix_embeddings(TINY_VLM, P, "fp32", 3 + i)).cuda() for i, P in enumerate(lens)]
    kc = [torch.zeros((TINY_VLM.n_layers, P, 1, TINY_VLM.head_dim), device="cuda") for P in lens]
    vc = [torch.zeros_like(k) for k in kc]
    jobs = [rosa.prefix_job(e, k, v, P) for e, k, v, P in zip(emb, kc, vc, lens)]
    sp, se = torch.cuda.Stream(), torch.cuda.Stream()
    pp = rosa.PrefixProducer(TINY_VLM, "fp32", w, 2, sum(lens), stream=sp.cuda_stream)
    pp.run(jobs)
    torch.cuda.synchronize()
    ref = [k.cpu().numpy().copy() for k in kc]
    ew = cached_weights(TINY_SHAPE, "fp32")
    reqs = make_requests(PRESETS["tiny"])
    ex = rosa.ActionExpert(TINY_SHAPE, "fp32", ew, rosa.capacity(2, 8, 16, 4, 200), stream=se.cuda_stream)
    dbt = rosa.DeviceBatch(reqs, "fp32")
    torch.cuda.synchronize()
    ex.generate(dbt.structs)
    torch.cuda.synchronize()
    alone = dbt.results()
    for _ in range(3):
        pp.run(jobs)
        ex.generate(dbt.structs)
    torch.cuda.synchronize()
    for k, r in zip(kc, ref):
        assert np.array_equal(k.cpu().numpy(), r)
    for x, y in zip(dbt.results(), alone):
        assert np.array_equal(x, y)
    pp.close()
    ex.close()
