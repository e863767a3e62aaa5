"""Python binding of the rosa C ABI (include/rosa.h, rosa_prefill.h, rosa_sched.h,
rosa_debug.h).

Argument marshalling only: every step of the computation runs in the HIP
library.  PyTorch supplies device memory and the stream.  The library must be
built (``python -m paper_2607_01088_amd.build``); loading fails loudly if it
is not.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librosa.so")

ROSA_OK, ROSA_E_INVALID, ROSA_E_CAPACITY, ROSA_E_NOMEM, ROSA_E_DEVICE, ROSA_E_UNSUPPORTED = range(6)
ROSA_BF16, ROSA_FP32 = 0, 1


class ModelConfig(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("d_mlp", C.c_int32),
                ("action_dim", C.c_int32), ("time_emb_dim", C.c_int32), ("rms_eps", C.c_float),
                ("dtype", C.c_int32), ("attention_layout", C.c_int32)]


_WEIGHT_FIELDS = ["w_in", "b_in", "w_t1", "b_t1", "w_t2", "b_t2", "w_mod", "b_mod", "w_qkv", "w_o",
                  "w_up", "w_down", "w_fmod", "b_fmod", "w_out", "b_out"]


class Weights(C.Structure):
    _fields_ = [(n, C.POINTER(C.c_float)) for n in _WEIGHT_FIELDS]


class Capacity(C.Structure):
    _fields_ = [("max_requests", C.c_int32), ("max_horizon", C.c_int32),
                ("max_action_tokens", C.c_int32), ("max_steps", C.c_int32),
                ("max_prefix_tokens", C.c_int64)]


class Request(C.Structure):
    _fields_ = [("prefix_k", C.c_void_p), ("prefix_v", C.c_void_p), ("noise", C.c_void_p),
                ("actions", C.c_void_p), ("prefix_len", C.c_int32), ("horizon", C.c_int32),
                ("num_steps", C.c_int32), ("start_step", C.c_int32)]


class S1Outcome(C.Structure):
    _fields_ = [("batch", C.c_int32), ("feasible", C.c_int32), ("throughput_hz", C.c_double),
                ("action_rate_hz", C.c_double), ("latency_mean_ms", C.c_double),
                ("latency_p50_ms", C.c_double), ("latency_p99_ms", C.c_double)]

    def as_dict(self) -> Dict[str, float]:
        return {n: getattr(self, n) for n, _ in self._fields_}


class VlmConfig(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("d_mlp", C.c_int32),
                ("rms_eps", C.c_float), ("dtype", C.c_int32), ("cache_form", C.c_int32),
                ("head_layers", C.c_int32), ("rope_base", C.c_float)]


_VLM_WEIGHT_FIELDS = ["w_qkv", "w_o", "w_up", "w_down", "w_ctx"]
ROSA_CACHE_PER_LAYER, ROSA_CACHE_CONTEXT = 0, 1


class VlmWeights(C.Structure):
    _fields_ = [(n, C.POINTER(C.c_float)) for n in _VLM_WEIGHT_FIELDS]


class PrefixJob(C.Structure):
    _fields_ = [("embeddings", C.c_void_p), ("prefix_k", C.c_void_p), ("prefix_v", C.c_void_p),
                ("prefix_len", C.c_int32), ("causal_len", C.c_int32)]


class RatePoint(C.Structure):
    _fields_ = [("rate_hz", C.c_double), ("mean_ms", C.c_double), ("slo_ms", C.c_double)]


class ConfigProfile(C.Structure):
    _fields_ = [("batch", C.c_int32), ("n_points", C.c_int32), ("points", C.POINTER(RatePoint))]


class ModelProfile(C.Structure):
    _fields_ = [("role", C.c_int32), ("max_streams", C.c_int32), ("deadline_ms", C.c_double),
                ("rate_per_robot_hz", C.c_double), ("n_configs", C.c_int32), ("reserved", C.c_int32),
                ("configs", C.POINTER(ConfigProfile))]


class Fleet(C.Structure):
    _fields_ = [("robots", C.c_int32), ("servers", C.c_int32), ("t_act_ms", C.c_double), ("horizon", C.c_int32),
                ("reserved", C.c_int32), ("eps_hz", C.c_double)]


class ServerPlan(C.Structure):
    _fields_ = [("model", C.c_int32), ("batch", C.c_int32), ("streams", C.c_int32), ("reserved", C.c_int32),
                ("mean_ms", C.c_double), ("slo_ms", C.c_double)]


class FleetSchedule(C.Structure):
    _fields_ = [("feasible", C.c_int32), ("obligation_servers", C.c_int32), ("goal_servers", C.c_int32),
                ("steps", C.c_int32), ("f_hz", C.c_double), ("l_s1_ms", C.c_double), ("l_s2_ms", C.c_double),
                ("f_loop_hz", C.c_double)]


ROSA_ROLE_S1, ROSA_ROLE_S2, ROSA_ROLE_OBLIGATION = 0, 1, 2


class RosaError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"rosa status {status}: {msg}")
        self.status = status


_lib = None


def load(path: Optional[str] = None) -> C.CDLL:
    """Load the built library (raises if it has not been built): `path`, else
    $ROSA_LIB_PATH (another build, e.g. the sanitized one), else the in-tree
    librosa.so."""
    global _lib
    if _lib is not None:
        return _lib
    p = path or os.environ.get("ROSA_LIB_PATH") or _LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"rosa HIP library not built: {p} is missing "
                           "(run python -m paper_2607_01088_amd.build)")
    lib = C.CDLL(p)
    vp, i32, i64 = C.c_void_p, C.c_int32, C.c_int64
    lib.rosa_batch_create.argtypes = [C.POINTER(ModelConfig), C.POINTER(Weights), C.POINTER(Capacity), vp,
                                      C.POINTER(vp)]
    lib.rosa_batch_create.restype = C.c_int
    lib.rosa_generate_actions.argtypes = [vp, C.POINTER(Request), i32]
    lib.rosa_generate_actions.restype = C.c_int
    lib.rosa_generate_steps.argtypes = [vp, C.POINTER(Request), i32, i32]
    lib.rosa_generate_steps.restype = C.c_int
    lib.rosa_destroy.argtypes = [vp]
    lib.rosa_destroy.restype = None
    lib.rosa_status_string.argtypes = [C.c_int]
    lib.rosa_status_string.restype = C.c_char_p
    lib.rosa_last_error.argtypes = [vp]
    lib.rosa_last_error.restype = C.c_char_p
    lib.rosa_debug_plan.argtypes = [C.POINTER(ModelConfig), C.POINTER(Capacity), C.POINTER(Request), i32,
                                    C.POINTER(i32), C.POINTER(i32), C.POINTER(i32), C.POINTER(i32)]
    lib.rosa_debug_plan.restype = C.c_int
    lib.rosa_attention_noalloc.argtypes = [C.POINTER(ModelConfig), C.POINTER(Request), i32, i32, vp, vp, vp]
    lib.rosa_attention_noalloc.restype = C.c_int
    lib.rosa_debug_plan_lanes.argtypes = [C.POINTER(ModelConfig), C.POINTER(Capacity), C.POINTER(Request), i32, i32,
                                          C.POINTER(i32)]
    lib.rosa_debug_plan_lanes.restype = C.c_int
    lib.rosa_debug_attn_lists.argtypes = [C.POINTER(ModelConfig), C.POINTER(Capacity), C.POINTER(Request), i32, i32,
                                          C.POINTER(i32), C.POINTER(i32), C.POINTER(i32), C.POINTER(i32),
                                          C.POINTER(i32)]
    lib.rosa_debug_attn_lists.restype = C.c_int
    lib.rosa_debug_mfma_peak.argtypes = [i32, C.POINTER(C.c_double)]
    lib.rosa_debug_mfma_peak.restype = C.c_int
    lib.rosa_debug_time_conditioning.argtypes = [vp, C.POINTER(C.c_float), i32, vp]
    lib.rosa_debug_time_conditioning.restype = C.c_int
    lib.rosa_debug_attention.argtypes = [vp, C.POINTER(Request), i32, i32, vp, vp]
    lib.rosa_debug_attention.restype = C.c_int
    lib.rosa_debug_gemm.argtypes = [vp, i32, i32, vp, i32, vp, vp]
    lib.rosa_debug_gemm.restype = C.c_int
    lib.rosa_debug_set_lanes.argtypes = [vp, i32]
    lib.rosa_debug_set_lanes.restype = C.c_int
    lib.rosa_debug_gemm_config.argtypes = [vp, i32, C.POINTER(i32)]
    lib.rosa_debug_gemm_config.restype = C.c_int
    lib.rosa_debug_set_profiling.argtypes = [vp, i32]
    lib.rosa_debug_set_profiling.restype = C.c_int
    lib.rosa_debug_get_profile.argtypes = [vp, C.POINTER(C.c_char_p), C.POINTER(i64), C.POINTER(C.c_double),
                                           i32, C.POINTER(i32)]
    lib.rosa_debug_get_profile.restype = C.c_int
    lib.rosa_s1_simulate.argtypes = [i32, i32, C.c_double, C.c_double, i32, C.POINTER(S1Outcome)]
    lib.rosa_s1_simulate.restype = C.c_int
    lib.rosa_s1_select_batch.argtypes = [C.POINTER(i32), C.POINTER(C.c_double), i32, i32, C.c_double, C.c_double,
                                         i32, C.POINTER(i32), C.POINTER(S1Outcome)]
    lib.rosa_s1_select_batch.restype = C.c_int
    lib.rosa_prefill_create.argtypes = [C.POINTER(VlmConfig), C.POINTER(VlmWeights), i32, i64, vp, C.POINTER(vp)]
    lib.rosa_prefill_create.restype = C.c_int
    lib.rosa_prefill_run.argtypes = [vp, C.POINTER(PrefixJob), i32]
    lib.rosa_prefill_run.restype = C.c_int
    lib.rosa_prefill_destroy.argtypes = [vp]
    lib.rosa_prefill_destroy.restype = None
    lib.rosa_prefill_last_error.argtypes = [vp]
    lib.rosa_prefill_last_error.restype = C.c_char_p
    lib.rosa_debug_prefill_set_profiling.argtypes = [vp, i32]
    lib.rosa_debug_prefill_set_profiling.restype = C.c_int
    lib.rosa_debug_prefill_gemm_config.argtypes = [vp, i32, C.POINTER(i32)]
    lib.rosa_debug_prefill_gemm_config.restype = C.c_int
    lib.rosa_debug_prefill_get_profile.argtypes = [vp, C.POINTER(C.c_char_p), C.POINTER(i64),
                                                   C.POINTER(C.c_double), i32, C.POINTER(i32)]
    lib.rosa_debug_prefill_get_profile.restype = C.c_int
    lib.rosa_rate_profile.argtypes = [i32, C.c_double, i32, i32, C.c_uint64, C.c_double, C.POINTER(RatePoint)]
    lib.rosa_rate_profile.restype = C.c_int
    lib.rosa_schedule_homogeneous.argtypes = [C.POINTER(Fleet), C.POINTER(ModelProfile), i32,
                                              C.POINTER(FleetSchedule), C.POINTER(ServerPlan)]
    lib.rosa_schedule_homogeneous.restype = C.c_int
    _lib = lib
    return lib


def model_config(shape, dtype: str) -> ModelConfig:
    return ModelConfig(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                       shape.d_mlp, shape.action_dim, shape.time_emb_dim, shape.rms_eps,
                       ROSA_BF16 if dtype == "bf16" else ROSA_FP32, getattr(shape, "attention_layout", 0))


def capacity(max_requests: int, max_horizon: int, max_action_tokens: int, max_steps: int,
             max_prefix_tokens: int) -> Capacity:
    return Capacity(max_requests, max_horizon, max_action_tokens, max_steps, max_prefix_tokens)


def _f32_ptr(a: np.ndarray):
    return a.ctypes.data_as(C.POINTER(C.c_float))


def request_struct(prefix_k, prefix_v, noise, actions, P: int, H: int, K: int, start_step: int = 0) -> Request:
    """Build a request from torch device tensors (or raw integer device pointers)."""
    def ptr(t):
        if t is None:
            return None
        return t if isinstance(t, int) else t.data_ptr()
    return Request(ptr(prefix_k), ptr(prefix_v), ptr(noise), ptr(actions), P, H, K, start_step)


def request_array(reqs: Sequence[Request]):
    arr = (Request * max(1, len(reqs)))()
    for i, r in enumerate(reqs):
        arr[i] = r
    return arr


def plan(shape, dtype: str, cap: Capacity, reqs: Sequence[Request]):
    """Host-only planning (rosa_debug_plan): (status, order, tok_off, m_k, counts)."""
    lib = load()
    cfg = model_config(shape, dtype)
    n = len(reqs)
    arr = request_array(reqs)
    order = (C.c_int32 * max(1, n))()
    tok = (C.c_int32 * max(1, n))()
    mk = (C.c_int32 * max(1, cap.max_steps))()
    counts = (C.c_int32 * 4)()
    st = lib.rosa_debug_plan(C.byref(cfg), C.byref(cap), arr, n, order, tok, mk, counts)
    return st, list(order)[:n], list(tok)[:n], list(mk)[:cap.max_steps], list(counts)


def attention_noalloc(shape, dtype: str, reqs: Sequence[Request], layer: int, qkv, o,
                      stream: Optional[int] = None) -> int:
    """rosa_attention_noalloc (no handle, no allocation) on torch tensors qkv and o;
    returns the status."""
    import torch
    lib = load()
    cfg = model_config(shape, dtype)
    if stream is None:
        stream = torch.cuda.current_stream().cuda_stream
    return lib.rosa_attention_noalloc(C.byref(cfg), request_array(reqs), len(reqs), layer, C.c_void_p(qkv.data_ptr()),
                                      C.c_void_p(o.data_ptr()), C.c_void_p(stream))


def last_error_global() -> str:
    """rosa_last_error(NULL): detail of the last failure of a handle-free call."""
    return load().rosa_last_error(None).decode()


def plan_lanes(shape, dtype: str, cap: Capacity, reqs: Sequence[Request], lanes: int):
    """Host-only lane assignment (rosa_debug_plan_lanes): (status, lane of each request)."""
    lib = load()
    cfg = model_config(shape, dtype)
    n = len(reqs)
    out = (C.c_int32 * max(1, n))()
    st = lib.rosa_debug_plan_lanes(C.byref(cfg), C.byref(cap), request_array(reqs), n, lanes, out)
    return st, list(out)[:n]


def attn_lists(shape, cap: Capacity, reqs: Sequence[Request], n_items: int):
    """Host-only attention launch lists of a bf16 call (rosa_debug_attn_lists):
    (status, n_blocks, item of each entry, next of each entry, cost of each item)."""
    lib = load()
    cfg = model_config(shape, "bf16")
    n = len(reqs)
    arr = request_array(reqs)
    nb, ne = C.c_int32(0), C.c_int32(0)
    st = lib.rosa_debug_attn_lists(C.byref(cfg), C.byref(cap), arr, n, 0, C.byref(nb), C.byref(ne), None, None, None)
    if st not in (ROSA_OK, ROSA_E_CAPACITY):
        return st, 0, [], [], []
    m = max(1, ne.value)
    item_of, nxt = (C.c_int32 * m)(), (C.c_int32 * m)()
    cost = (C.c_int32 * max(1, n_items))()
    st = lib.rosa_debug_attn_lists(C.byref(cfg), C.byref(cap), arr, n, m, C.byref(nb), C.byref(ne), item_of, nxt, cost)
    return st, nb.value, list(item_of)[:ne.value], list(nxt)[:ne.value], list(cost)[:n_items]


def mfma_peak(device: int = 0) -> float:
    """Attainable dense bf16 MFMA rate of the GPU in TFLOP/s (rosa_debug_mfma_peak)."""
    lib = load()
    v = C.c_double(0.0)
    st = lib.rosa_debug_mfma_peak(device, C.byref(v))
    if st != ROSA_OK:
        raise RosaError(st, "rosa_debug_mfma_peak failed")
    return v.value


def s1_simulate(robots: int, batch: int, batch_ms: float, t_act_ms: float, n_batches: int = 256) -> Dict[str, float]:
    """Closed-loop simulation of one System-1 worker (rosa_s1_simulate)."""
    lib = load()
    o = S1Outcome()
    st = lib.rosa_s1_simulate(robots, batch, batch_ms, t_act_ms, n_batches, C.byref(o))
    if st != ROSA_OK:
        raise RosaError(st, "rosa_s1_simulate: invalid arguments")
    return o.as_dict()


def s1_select_batch(batch_sizes: Sequence[int], batch_ms: Sequence[float], robots: int, t_act_ms: float,
                    slo_ms: float, n_batches: int = 256):
    """Batch-size choice from a measured profile (rosa_s1_select_batch):
    returns (index or None, list of outcome dicts in input order)."""
    lib = load()
    n = len(batch_sizes)
    sizes = (C.c_int32 * max(1, n))(*batch_sizes)
    ms = (C.c_double * max(1, n))(*batch_ms)
    outs = (S1Outcome * max(1, n))()
    best = C.c_int32(-2)
    st = lib.rosa_s1_select_batch(sizes, ms, n, robots, t_act_ms, slo_ms, n_batches, C.byref(best), outs)
    if st != ROSA_OK:
        raise RosaError(st, "rosa_s1_select_batch: invalid arguments")
    return (None if best.value < 0 else best.value), [outs[i].as_dict() for i in range(n)]


def rate_profile(batch: int, batch_ms: float, n_rates: int = 10, n_requests: int = 4000, seed: int = 1,
                 pct: float = 0.99) -> List[tuple]:
    """rosa_rate_profile: [(rate_hz, mean_ms, slo_ms)] of one batch size."""
    lib = load()
    out = (RatePoint * n_rates)()
    st = lib.rosa_rate_profile(batch, batch_ms, n_rates, n_requests, seed, pct, out)
    if st != ROSA_OK:
        raise RosaError(st, "rosa_rate_profile: invalid arguments")
    return [(p.rate_hz, p.mean_ms, p.slo_ms) for p in out]


def schedule_homogeneous(fleet: Dict, models: Sequence[Dict]) -> Dict:
    """rosa_schedule_homogeneous.  fleet: robots, servers, t_act_ms, horizon,
    eps_hz.  models: dicts with role (ROSA_ROLE_*), deadline_ms, profile
    [(batch, [(rate, mean, slo), ...])], optional max_streams and
    rate_per_robot_hz.  Returns the schedule with assignment
    [(model, (batch, streams, mean_ms, slo_ms))]."""
    lib = load()
    keep = []
    mp = (ModelProfile * len(models))()
    for i, m in enumerate(models):
        cps = (ConfigProfile * len(m["profile"]))()
        for j, (batch, pts) in enumerate(m["profile"]):
            arr = (RatePoint * len(pts))(*[RatePoint(*p) for p in pts])
            keep.append(arr)
            cps[j] = ConfigProfile(batch, len(pts), arr)
        keep.append(cps)
        mp[i] = ModelProfile(m["role"], m.get("max_streams", 0), m["deadline_ms"], m.get("rate_per_robot_hz", 0.0),
                             len(m["profile"]), 0, cps)
    fl = Fleet(fleet["robots"], fleet["servers"], fleet["t_act_ms"], fleet.get("horizon", 1), 0, fleet["eps_hz"])
    out = FleetSchedule()
    plans = (ServerPlan * fleet["servers"])()
    st = lib.rosa_schedule_homogeneous(C.byref(fl), mp, len(models), C.byref(out), plans)
    if st != ROSA_OK:
        raise RosaError(st, "rosa_schedule_homogeneous: invalid arguments")
    n = out.obligation_servers + out.goal_servers if out.feasible else 0
    return {"feasible": bool(out.feasible), "f_hz": out.f_hz, "l_s1_ms": out.l_s1_ms, "l_s2_ms": out.l_s2_ms,
            "f_loop_hz": out.f_loop_hz, "obligation_servers": out.obligation_servers,
            "goal_servers": out.goal_servers, "steps": out.steps,
            "assignment": [(plans[i].model, (plans[i].batch, plans[i].streams, plans[i].mean_ms, plans[i].slo_ms))
                           for i in range(n)]}


class ActionExpert:
    """A rosa_batch handle: the action expert's weights on the GPU plus workspaces."""

    def __init__(self, shape, dtype: str, weights: Dict[str, np.ndarray], cap: Capacity,
                 stream: Optional[int] = None):
        import torch
        self.lib = load()
        self.shape, self.dtype, self.cap = shape, dtype, cap
        self._cfg = model_config(shape, dtype)
        self._host = {k: np.ascontiguousarray(weights[k], dtype=np.float32) for k in _WEIGHT_FIELDS}
        w = Weights(*[_f32_ptr(self._host[k]) for k in _WEIGHT_FIELDS])
        if stream is None:
            stream = torch.cuda.current_stream().cuda_stream
        self.stream = stream
        h = C.c_void_p()
        st = self.lib.rosa_batch_create(C.byref(self._cfg), C.byref(w), C.byref(cap), C.c_void_p(stream),
                                        C.byref(h))
        self._host = None   # the library copied what it needs
        if st != ROSA_OK:
            raise RosaError(st, self.lib.rosa_last_error(None).decode())
        self.handle = h

    def _check(self, st: int):
        if st != ROSA_OK:
            raise RosaError(st, self.lib.rosa_last_error(self.handle).decode())

    def generate(self, reqs: Sequence[Request]) -> int:
        """Enqueue rosa_generate_actions; returns the status (raises on error)."""
        arr = request_array(reqs)
        st = self.lib.rosa_generate_actions(self.handle, arr, len(reqs))
        self._check(st)
        return st

    def generate_steps(self, reqs: Sequence[Request], max_steps: int) -> int:
        """Enqueue rosa_generate_steps (each request runs at most max_steps of
        its remaining Euler steps from its start_step); raises on error."""
        arr = request_array(reqs)
        st = self.lib.rosa_generate_steps(self.handle, arr, len(reqs), max_steps)
        self._check(st)
        return st

    def generate_status(self, reqs: Sequence[Request]) -> int:
        """Like generate but returns the status instead of raising."""
        arr = request_array(reqs)
        return self.lib.rosa_generate_actions(self.handle, arr, len(reqs))

    def time_conditioning(self, taus: Sequence[float], out) -> None:
        t = (C.c_float * len(taus))(*taus)
        self._check(self.lib.rosa_debug_time_conditioning(self.handle, t, len(taus), out.data_ptr()))

    def attention(self, reqs: Sequence[Request], layer: int, qkv, o) -> None:
        arr = request_array(reqs)
        self._check(self.lib.rosa_debug_attention(self.handle, arr, len(reqs), layer, qkv.data_ptr(),
                                                  o.data_ptr()))

    def gemm(self, which: int, layer: int, a, M: int, out, gate=None) -> None:
        self._check(self.lib.rosa_debug_gemm(self.handle, which, layer, a.data_ptr(), M, out.data_ptr(),
                                             None if gate is None else gate.data_ptr()))

    def set_lanes(self, n: int) -> None:
        """Number of concurrent sub-batches (streams) per call."""
        self._check(self.lib.rosa_debug_set_lanes(self.handle, n))

    def gemm_config(self, cfg: int) -> int:
        """Force the projection block configuration (-1: cost model); returns
        the number of configurations."""
        n = C.c_int32()
        self._check(self.lib.rosa_debug_gemm_config(self.handle, cfg, C.byref(n)))
        return n.value

    def set_profiling(self, enable: bool) -> None:
        self._check(self.lib.rosa_debug_set_profiling(self.handle, 1 if enable else 0))

    def profile(self) -> Dict[str, tuple]:
        n = 32
        names = (C.c_char_p * n)()
        launches = (C.c_int64 * n)()
        ms = (C.c_double * n)()
        cnt = C.c_int32()
        self._check(self.lib.rosa_debug_get_profile(self.handle, names, launches, ms, n, C.byref(cnt)))
        return {names[i].decode(): (int(launches[i]), float(ms[i])) for i in range(cnt.value)}

    def close(self) -> None:
        if getattr(self, "handle", None):
            self.lib.rosa_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def vlm_config(shape, dtype: str, head_layers: int = 0) -> VlmConfig:
    """head_layers > 0: the context cache form for a head of that many layers."""
    return VlmConfig(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                     shape.d_mlp, shape.rms_eps, ROSA_BF16 if dtype == "bf16" else ROSA_FP32,
                     ROSA_CACHE_CONTEXT if head_layers > 0 else ROSA_CACHE_PER_LAYER, head_layers,
                     float(getattr(shape, "rope_base", 0.0)))


def prefix_job(embeddings, prefix_k, prefix_v, P: int, causal_len: int = 0) -> PrefixJob:
    """A prefix-producer job from torch device tensors (or raw integer device
    pointers); causal_len: the job's trailing causal segment (0: none)."""
    def ptr(t):
        return t if isinstance(t, int) else t.data_ptr()
    return PrefixJob(ptr(embeddings), ptr(prefix_k), ptr(prefix_v), P, causal_len)


class PrefixProducer:
    """A rosa_prefill handle: the VLM backbone's weights on the GPU plus workspaces."""

    def __init__(self, shape, dtype: str, weights: Dict[str, np.ndarray], max_jobs: int, max_tokens: int,
                 stream: Optional[int] = None, context_weights: Optional[np.ndarray] = None):
        """context_weights ([L_e][d][2 n_kv hd]): the context cache form for a
        cross-attending head of L_e layers; None: per-layer caches."""
        import torch
        self.lib = load()
        self.shape, self.dtype = shape, dtype
        head_layers = 0 if context_weights is None else int(context_weights.shape[0])
        self._cfg = vlm_config(shape, dtype, head_layers)
        host = {k: np.ascontiguousarray(weights[k], dtype=np.float32) for k in _VLM_WEIGHT_FIELDS if k != "w_ctx"}
        if context_weights is not None:
            host["w_ctx"] = np.ascontiguousarray(context_weights, dtype=np.float32)
        w = VlmWeights(*[_f32_ptr(host[k]) if k in host else None for k in _VLM_WEIGHT_FIELDS])
        if stream is None:
            stream = torch.cuda.current_stream().cuda_stream
        self.stream = stream
        h = C.c_void_p()
        st = self.lib.rosa_prefill_create(C.byref(self._cfg), C.byref(w), max_jobs, max_tokens, C.c_void_p(stream),
                                          C.byref(h))
        del host   # the library copied what it needs
        if st != ROSA_OK:
            raise RosaError(st, self.lib.rosa_prefill_last_error(None).decode())
        self.handle = h

    def _check(self, st: int):
        if st != ROSA_OK:
            raise RosaError(st, self.lib.rosa_prefill_last_error(self.handle).decode())

    def run_status(self, jobs: Sequence[PrefixJob]) -> int:
        arr = (PrefixJob * max(1, len(jobs)))(*jobs)
        return self.lib.rosa_prefill_run(self.handle, arr, len(jobs))

    def run(self, jobs: Sequence[PrefixJob]) -> None:
        """Enqueue rosa_prefill_run; raises on error."""
        self._check(self.run_status(jobs))

    def set_profiling(self, enable: bool) -> None:
        self._check(self.lib.rosa_debug_prefill_set_profiling(self.handle, 1 if enable else 0))

    def gemm_config(self, cfg: int) -> int:
        """Force the projection block configuration (-1: cost model); returns
        the number of configurations."""
        n = C.c_int32()
        self._check(self.lib.rosa_debug_prefill_gemm_config(self.handle, cfg, C.byref(n)))
        return n.value

    def profile(self) -> Dict[str, tuple]:
        n = 16
        names = (C.c_char_p * n)()
        launches = (C.c_int64 * n)()
        ms = (C.c_double * n)()
        cnt = C.c_int32()
        self._check(self.lib.rosa_debug_prefill_get_profile(self.handle, names, launches, ms, n, C.byref(cnt)))
        return {names[i].decode(): (int(launches[i]), float(ms[i])) for i in range(cnt.value)}

    def close(self) -> None:
        if getattr(self, "handle", None):
            self.lib.rosa_prefill_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------- device upload helpers

def to_device_kv(arr: np.ndarray, dtype: str, device="cuda"):
    """Prefix KV array (uint16 bf16 bits or float32) -> torch device tensor."""
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32))
    return t.to(device)


class DeviceBatch:
    """A list of requests uploaded to the GPU (prefix KV resident), with output
    buffers, and the request structs that point at them."""

    def __init__(self, requests, dtype: str, device="cuda"):
        import torch
        self.k, self.v, self.noise, self.actions, self.structs = [], [], [], [], []
        for r in requests:
            k = to_device_kv(r.prefix_k, dtype, device) if r.prefix_len > 0 else None
            v = to_device_kv(r.prefix_v, dtype, device) if r.prefix_len > 0 else None
            nz = torch.from_numpy(np.ascontiguousarray(r.noise, dtype=np.float32)).to(device)
            out = torch.full_like(nz, float("nan"))
            self.k.append(k); self.v.append(v); self.noise.append(nz); self.actions.append(out)
            self.structs.append(request_struct(k, v, nz, out, r.prefix_len, r.horizon, r.steps))

    def results(self) -> List[np.ndarray]:
        return [a.cpu().numpy() for a in self.actions]
