"""The whole System-1 path at full size on the GPU: the PaliGemma-sized
backbone fills 32 robots' prefix caches (rosa_prefill_run) and the pi0-shaped
expert generates their action chunks from those caches
(rosa_generate_actions), with no host round trip in between; the shortest
request is checked against the oracle chain (backbone, then expert)."""
import numpy as np
import pytest

from oracle import OracleModel, prefill
from synthetic import PI0_SHAPE, PI0_VLM, make_prefix_embeddings, make_vlm_weights, prefill_lengths
from tests.helpers import cached_weights, rel_l2

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.mark.timeout(600)
def test_prefill_then_generate_full_size():
    from paper_2607_01088_amd import rosa
    lens = prefill_lengths()
    H, K, A = 50, 10, PI0_SHAPE.action_dim
    vw = make_vlm_weights(PI0_VLM, "bf16")
    xs = [make_prefix_embeddings(PI0_VLM, P, "bf16", 4000 + i) for i, P in enumerate(lens)]
    emb = [torch.from_numpy(x).to(torch.bfloat16).cuda() for x in xs]
    kc = [torch.full((PI0_SHAPE.n_layers, P, 1, 256), float("nan"), dtype=torch.bfloat16, device="cuda") for P in lens]
    vc = [torch.full_like(k, float("nan")) for k in kc]
    pp = rosa.PrefixProducer(PI0_VLM, "bf16", vw, len(lens), sum(lens))
    pp.run([rosa.prefix_job(e, k, v, P) for e, k, v, P in zip(emb, kc, vc, lens)])
    rng = np.random.default_rng(5)
    noise = [rng.standard_normal((H, A)).astype(np.float32) for _ in lens]
    nz = [torch.from_numpy(n).cuda() for n in noise]
    out = [torch.full_like(n, float("nan")) for n in nz]
    ew = cached_weights(PI0_SHAPE, "bf16")
    ex = rosa.ActionExpert(PI0_SHAPE, "bf16", ew, rosa.capacity(len(lens), H, H * len(lens), K, sum(lens)))
    ex.generate([rosa.request_struct(k, v, n, o, P, H, K) for k, v, n, o, P in zip(kc, vc, nz, out, lens)])
    torch.cuda.synchronize()
    got = [o.cpu().numpy() for o in out]
    assert all(np.isfinite(g).all() for g in got)
    i = int(np.argmin(lens))
    Kc, Vc = prefill(xs[i], vw, PI0_VLM)
    ref = OracleModel(ew, PI0_SHAPE).generate_chunk(noise[i], K, Kc, Vc)
    err = rel_l2(got[i], ref)
    print(f"pipeline request {i} P={lens[i]}: rel-L2 {err:.2e}", flush=True)
    assert err <= 1e-2
    pp.close()
    ex.close()
