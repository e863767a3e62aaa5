"""Shared test helpers (no method arithmetic here: comparisons and plumbing)."""
from __future__ import annotations

import functools
import os
import re
from typing import List, Sequence

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _shape(**kw):
    from synthetic import ModelShape
    return ModelShape(**kw)


# Whole-call and attention tests at the head widths the presets do not use:
# grouped-query attention with two query heads per KV head at head_dim 64,
# plain multi-head attention at head_dim 128.
HD64_SHAPE = _shape(n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=2, head_dim=64, d_mlp=512, action_dim=7,
                    time_emb_dim=128)
HD128_SHAPE = _shape(n_layers=3, d_model=384, n_q_heads=3, n_kv_heads=3, head_dim=128, d_mlp=768, action_dim=14,
                     time_emb_dim=64)


def declared_functions() -> List[str]:
    """Every function the public headers declare."""
    names = []
    for h in ["rosa.h", "rosa_debug.h", "rosa_sched.h", "rosa_prefill.h"]:
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names += re.findall(r"\b(rosa_[a-z0-9_]+)\s*\(", src)
    return sorted(set(names))


def rel_l2(a: np.ndarray, b: np.ndarray) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (den if den > 0 else 1.0))


@functools.lru_cache(maxsize=4)
def cached_weights(shape, dtype: str, seed: int = 0):
    from synthetic import make_weights
    return make_weights(shape, dtype, seed)


def cap_for(requests, max_requests=None, max_steps=None):
    from paper_2607_01088_amd import rosa
    n = len(requests)
    return rosa.capacity(max_requests or max(1, n), max(r.horizon for r in requests),
                         sum(r.horizon for r in requests), max_steps or max(r.steps for r in requests),
                         sum(r.prefix_len for r in requests))
