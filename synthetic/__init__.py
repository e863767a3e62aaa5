"""Seeded synthetic inputs for batched action-chunk generation.

This module only draws random numbers and lays them out: model shapes, weights,
per-request prefix KV caches, initial action noise, prefix lengths, horizons and
step counts.  It holds none of the method's arithmetic, so both the CPU oracle
and the GPU library can consume the same inputs without sharing any code.

The workloads stand in for the paper's System-1 action model serving a fleet of
robots (Sec. 3.2 and 3.4.1: requests from many robots are batched into one
action-model call; Sec. 4.3, the System-1 batching ablation).  The paper evaluates GR00T N1.6
and pi0.5 on real observations; those weights and observations are not
available, so every tensor here is synthetic with the shapes of a pi0-style
action expert (18 layers, width 1024, 8 query heads sharing one 256-wide KV
head, GELU MLP of width 4096, 32-dim actions).

Random-draw recipe (fixed, so any request can be regenerated alone):

* ``numpy.random.Generator(PCG64)``; the master ``SeedSequence(seed)`` is
  spawned into children ``[weights, metadata, request_0, request_1, ...]``.
* Weights: every matrix is N(0, 0.02^2); every bias is 0.  Tensors are drawn in
  the order of ``WEIGHT_ORDER`` from the weights child.
* Metadata (prefix lengths, horizons, step counts) comes from the metadata
  child, in that order; integer ranges include both ends.
* Request r draws, from its own child, prefix K for all layers, then prefix V
  for all layers (each ``[L][P][n_kv][hd]``, N(0,1)), then noise ``[H][A]``
  (N(0,1)).
* In bf16 mode weights and prefix KV are rounded to bfloat16 with
  round-to-nearest-even; noise stays float32.  Both sides see the same values.
"""
from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence

import numpy as np

__all__ = [
    "ModelShape", "Preset", "RequestData", "PRESETS", "WEIGHT_ORDER",
    "TINY_SHAPE", "PI0_SHAPE", "TINY_ALT_SHAPE", "PI0_ALT_SHAPE", "bf16_round", "bf16_bits", "bits_to_f32",
    "make_weights", "make_metadata", "make_request", "make_requests",
    "weight_shapes", "VlmShape", "TINY_VLM", "PI0_VLM", "VLM_WEIGHT_ORDER", "vlm_weight_shapes",
    "make_vlm_weights", "make_prefix_embeddings", "prefill_lengths", "make_context_weights",
]


@dataclasses.dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_mlp: int
    action_dim: int
    time_emb_dim: int
    rms_eps: float = 1e-6
    # 0: joint attention over [prefix ; own actions] in every layer (pi0-style);
    # 1: alternating, even layers cross-attend to the prefix only and odd
    #    layers self-attend to the request's own actions only (GR00T-style DiT).
    attention_layout: int = 0

    @property
    def qkv_dim(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim


TINY_SHAPE = ModelShape(n_layers=2, d_model=128, n_q_heads=4, n_kv_heads=1, head_dim=32,
                        d_mlp=512, action_dim=7, time_emb_dim=128)
PI0_SHAPE = ModelShape(n_layers=18, d_model=1024, n_q_heads=8, n_kv_heads=1, head_dim=256,
                       d_mlp=4096, action_dim=32, time_emb_dim=1024)
# The same sizes with the alternating cross-/self-attention layout.
TINY_ALT_SHAPE = dataclasses.replace(TINY_SHAPE, attention_layout=1)
PI0_ALT_SHAPE = dataclasses.replace(PI0_SHAPE, attention_layout=1)


@dataclasses.dataclass(frozen=True)
class Preset:
    """A named workload: model shape, dtype and how the batch is drawn."""
    name: str
    shape: ModelShape
    dtype: str                      # "bf16" or "fp32"
    batch: int
    prefix_lens: Optional[Sequence[int]] = None   # fixed list, else drawn
    prefix_range: Optional[Sequence[int]] = None  # (lo, hi) inclusive
    horizons: Sequence[int] = (50,)               # drawn uniformly from this set
    steps: Sequence[int] = (10,)                  # drawn uniformly from this set
    description: str = ""


PRESETS: Dict[str, Preset] = {
    p.name: p for p in [
        Preset("tiny", TINY_SHAPE, "fp32", 2, prefix_lens=(64, 96), horizons=(8,), steps=(4,),
               description="plumbing case: 2 requests, prefixes 64 and 96, horizon 8, 4 steps"),
        Preset("pi0_b1", PI0_SHAPE, "bf16", 1, prefix_lens=(816,), horizons=(50,), steps=(10,),
               description="one robot: prefix 816 = 3 images x 256 patches + 48 text tokens"),
        Preset("pi0_b32", PI0_SHAPE, "bf16", 32, prefix_range=(600, 1024), horizons=(50,), steps=(10,),
               description="32 robots, prefix lengths uniform in [600, 1024]"),
        Preset("factory_b256", PI0_SHAPE, "bf16", 256, prefix_range=(512, 1280), horizons=(16, 50),
               steps=(5, 10),
               description="factory fleet: 256 ragged requests, prefix U[512,1280], "
                           "horizon 16 or 50, 5 or 10 steps"),
        Preset("stress_b512", PI0_SHAPE, "bf16", 512, prefix_range=(1024, 2048), horizons=(50,),
               steps=(10,),
               description="large fleet, long context: 512 requests, prefix U[1024,2048]"),
    ]
}

WEIGHT_ORDER = ["w_in", "b_in", "w_t1", "b_t1", "w_t2", "b_t2", "w_mod", "b_mod",
                "w_qkv", "w_o", "w_up", "w_down", "w_fmod", "b_fmod", "w_out", "b_out"]


def weight_shapes(s: ModelShape) -> Dict[str, tuple]:
    """Host weight shapes, all row-major [in][out] (y = x @ W)."""
    L, d, A, dt = s.n_layers, s.d_model, s.action_dim, s.time_emb_dim
    return {
        "w_in": (A, d), "b_in": (d,),
        "w_t1": (dt, d), "b_t1": (d,), "w_t2": (d, d), "b_t2": (d,),
        "w_mod": (L, d, 6 * d), "b_mod": (L, 6 * d),
        "w_qkv": (L, d, s.qkv_dim), "w_o": (L, s.n_q_heads * s.head_dim, d),
        "w_up": (L, d, s.d_mlp), "w_down": (L, s.d_mlp, d),
        "w_fmod": (d, 2 * d), "b_fmod": (2 * d,), "w_out": (d, A), "b_out": (A,),
    }


# ---------------------------------------------------------------- bfloat16 helpers

def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)
    return r.astype(np.uint16)


def bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 values rounded to the nearest bfloat16, returned as float32."""
    return bits_to_f32(bf16_bits(x))


# ---------------------------------------------------------------- draws

def _children(seed: int, n_requests: int):
    ss = np.random.SeedSequence(seed)
    kids = ss.spawn(2 + n_requests)
    return kids[0], kids[1], kids[2:]


def make_weights(shape: ModelShape, dtype: str = "bf16", seed: int = 0, std: float = 0.02
                 ) -> Dict[str, np.ndarray]:
    """Weights as float32 arrays (bf16-representable values in bf16 mode)."""
    wss, _, _ = _children(seed, 0)
    rng = np.random.Generator(np.random.PCG64(wss))
    out = {}
    for name in WEIGHT_ORDER:
        shp = weight_shapes(shape)[name]
        if name.startswith("b_"):
            w = np.zeros(shp, dtype=np.float32)
        else:
            w = rng.standard_normal(shp, dtype=np.float32)
            w *= np.float32(std)
            if dtype == "bf16":
                w = bf16_round(w)
        out[name] = w
    return out


@dataclasses.dataclass
class RequestMeta:
    prefix_len: int
    horizon: int
    steps: int


def make_metadata(preset: Preset, seed: int = 0) -> List[RequestMeta]:
    _, mss, _ = _children(seed, preset.batch)
    rng = np.random.Generator(np.random.PCG64(mss))
    B = preset.batch
    if preset.prefix_lens is not None:
        P = np.asarray(preset.prefix_lens, dtype=np.int64)
    else:
        lo, hi = preset.prefix_range
        P = rng.integers(lo, hi, size=B, endpoint=True)
    H = rng.choice(np.asarray(preset.horizons), size=B) if len(preset.horizons) > 1 \
        else np.full(B, preset.horizons[0])
    K = rng.choice(np.asarray(preset.steps), size=B) if len(preset.steps) > 1 \
        else np.full(B, preset.steps[0])
    return [RequestMeta(int(P[i]), int(H[i]), int(K[i])) for i in range(B)]


@dataclasses.dataclass
class RequestData:
    """One robot request.  ``prefix_k``/``prefix_v`` are ``[L][P][n_kv][hd]``:
    uint16 bf16 bit patterns in bf16 mode, float32 in fp32 mode.  ``noise`` is
    float32 ``[H][A]``."""
    prefix_k: np.ndarray
    prefix_v: np.ndarray
    noise: np.ndarray
    prefix_len: int
    horizon: int
    steps: int
    dtype: str

    def prefix_f32(self, which: str) -> np.ndarray:
        a = self.prefix_k if which == "k" else self.prefix_v
        return bits_to_f32(a) if self.dtype == "bf16" else a


def _draw_request(shape: ModelShape, dtype: str, meta: RequestMeta, ss: np.random.SeedSequence
                  ) -> RequestData:
    rng = np.random.Generator(np.random.PCG64(ss))
    kv_shape = (shape.n_layers, meta.prefix_len, shape.n_kv_heads, shape.head_dim)
    k = rng.standard_normal(kv_shape, dtype=np.float32)
    v = rng.standard_normal(kv_shape, dtype=np.float32)
    noise = rng.standard_normal((meta.horizon, shape.action_dim), dtype=np.float32)
    if dtype == "bf16":
        k, v = bf16_bits(k), bf16_bits(v)
    return RequestData(k, v, noise, meta.prefix_len, meta.horizon, meta.steps, dtype)


def make_request(preset: Preset, r: int, seed: int = 0,
                 meta: Optional[List[RequestMeta]] = None) -> RequestData:
    """Regenerate request ``r`` of a preset alone (same values as in the batch)."""
    meta = meta if meta is not None else make_metadata(preset, seed)
    _, _, kids = _children(seed, preset.batch)
    return _draw_request(preset.shape, preset.dtype, meta[r], kids[r])


def make_requests(preset: Preset, seed: int = 0, indices: Optional[Sequence[int]] = None,
                  threads: int = 8) -> List[RequestData]:
    """Draw the batch (or a subset of it) with a thread pool; the values do not
    depend on the thread count."""
    meta = make_metadata(preset, seed)
    _, _, kids = _children(seed, preset.batch)
    idx = list(range(preset.batch)) if indices is None else list(indices)
    if threads <= 1 or len(idx) <= 1:
        return [_draw_request(preset.shape, preset.dtype, meta[r], kids[r]) for r in idx]
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return list(ex.map(lambda r: _draw_request(preset.shape, preset.dtype, meta[r], kids[r]), idx))


def custom_request(shape: ModelShape, dtype: str, prefix_len: int, horizon: int, steps: int,
                   seed: int) -> RequestData:
    """A request outside any preset (test edge cases: P = 0, H = 1, ...)."""
    return _draw_request(shape, dtype, RequestMeta(prefix_len, horizon, steps),
                         np.random.SeedSequence(seed))


# ---------------------------------------------------------------- vision-language prefix producer

@dataclasses.dataclass(frozen=True)
class VlmShape:
    """A VLM backbone whose per-layer keys and values are the action expert's
    prefix cache: same layer count, KV heads and head width as the expert."""
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_mlp: int
    rms_eps: float = 1e-6
    rope_base: float = 0.0      # > 1: rotary position embedding of queries and keys; 0: no positions

    @property
    def qkv_dim(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim


# Pairs with TINY_SHAPE (2 layers, 1 KV head of 32) and PI0_SHAPE (18 layers,
# 1 KV head of 256; a PaliGemma-sized backbone: width 2048, 8 heads, MLP 16384).
TINY_VLM = VlmShape(n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=1, head_dim=32, d_mlp=1024)
PI0_VLM = VlmShape(n_layers=18, d_model=2048, n_q_heads=8, n_kv_heads=1, head_dim=256, d_mlp=16384)

VLM_WEIGHT_ORDER = ["w_qkv", "w_o", "w_up", "w_down"]


def vlm_weight_shapes(s: VlmShape) -> Dict[str, tuple]:
    """Host weight shapes of the backbone, row-major [in][out] (y = x @ W)."""
    L, d = s.n_layers, s.d_model
    return {"w_qkv": (L, d, s.qkv_dim), "w_o": (L, s.n_q_heads * s.head_dim, d),
            "w_up": (L, d, s.d_mlp), "w_down": (L, s.d_mlp, d)}


def make_vlm_weights(shape: VlmShape, dtype: str = "bf16", seed: int = 1, std: float = 0.02,
                     threads: int = 16) -> Dict[str, np.ndarray]:
    """Backbone weights N(0, std^2); bf16-representable in bf16 mode.  The
    weights child of SeedSequence(seed) is spawned into one child per (tensor,
    layer), tensor-major in VLM_WEIGHT_ORDER, and each layer's matrix is drawn
    from its own child, so layers are drawn in parallel with the same values."""
    wss, _, _ = _children(seed, 0)
    L = shape.n_layers
    kids = wss.spawn(len(VLM_WEIGHT_ORDER) * L)
    shapes = vlm_weight_shapes(shape)
    out = {n: np.empty(shapes[n], dtype=np.float32) for n in VLM_WEIGHT_ORDER}

    def draw(job):
        ti, l = divmod(job, L)
        name = VLM_WEIGHT_ORDER[ti]
        rng = np.random.Generator(np.random.PCG64(kids[job]))
        w = rng.standard_normal(shapes[name][1:], dtype=np.float32)
        w *= np.float32(std)
        out[name][l] = bf16_round(w) if dtype == "bf16" else w

    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        list(ex.map(draw, range(len(VLM_WEIGHT_ORDER) * L)))
    return out


def make_prefix_embeddings(shape: VlmShape, prefix_len: int, dtype: str, seed: int) -> np.ndarray:
    """Input embeddings of one request's prefix tokens (image patches and text,
    already embedded), [P][d] N(0, 1), bf16-representable float32 in bf16 mode."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    x = rng.standard_normal((prefix_len, shape.d_model), dtype=np.float32)
    return bf16_round(x) if dtype == "bf16" else x


def prefill_lengths(n_jobs: int = 32, lo: int = 600, hi: int = 1024, seed: int = 11) -> List[int]:
    """Prefix lengths of a prefill batch: n_jobs draws, uniform on [lo, hi]
    inclusive, from numpy.random.default_rng(seed).  The default is the
    benchmarked batch: 32 robots' prefixes of a few camera images plus an
    instruction (600..1024 tokens, as the pi0_b32 preset)."""
    rng = np.random.default_rng(seed)
    return [int(p) for p in rng.integers(lo, hi + 1, size=n_jobs)]


def make_context_weights(shape: VlmShape, head_layers: int, dtype: str = "bf16", seed: int = 2,
                         std: float = 0.02) -> np.ndarray:
    """Context projection weights of a cross-attending action head:
    [head_layers][d][2 n_kv hd] (K columns, then V), N(0, std^2) from the
    weights child of SeedSequence(seed); bf16-representable in bf16 mode."""
    wss, _, _ = _children(seed, 0)
    rng = np.random.Generator(np.random.PCG64(wss))
    w = rng.standard_normal((head_layers, shape.d_model, 2 * shape.n_kv_heads * shape.head_dim), dtype=np.float32)
    w *= np.float32(std)
    return bf16_round(w) if dtype == "bf16" else w
