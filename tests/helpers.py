"""Shared test helpers (no method arithmetic here: comparisons and plumbing)."""
from __future__ import annotations

import functools
import os
import re
from typing import List, Sequence

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


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
