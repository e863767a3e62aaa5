"""CPU oracle for System-1 batch-size selection (test infrastructure only).

The paper's scheduler chooses a discrete System-1 batch size per server from
measured latency profiles (Sec. 3.4.1, batching decisions; Sec. 3.4.2, Step
2.1: per-server configurations from measured serving profiles; Sec. 4.3,
System-1 batching: larger batches raise throughput but add latency and
queueing, so the best size depends on load).  Robots run closed loop: wait for
the action chunk, execute it for t_act, send the next request, so the action
rate is bounded by 1 / (t_act + l_S1) (Sec. 3.4.2, Step 2.3).

The paper gives no queueing model for one worker; the reading taken here:
identical robots, all submitting at time 0; a FIFO queue (ties by robot
index); a batch starts when the worker is idle and b requests wait, takes the
b oldest and returns them all after the measured call latency T(b); a robot
resubmits t_act after its chunk returns; fewer robots than b means no batch
ever forms.  Statistics cover the second half of the simulated batches.

Pins (tests marked ``not gpu``): closed forms of the periodic regimes --
robots = b (latency T, rate 1 / (T + t_act)); robots = m b with
t_act >= (m - 1) T (no waiting); robots = m b with t_act < (m - 1) T (the
worker is always busy: throughput b / T, latency m T - t_act); a saturated
worker with robots not a multiple of b (throughput b / T); robots < b
(infeasible); an idle worker waiting for the b-th request of a batch; the
nearest-rank percentile against NumPy's inverted-CDF percentile.  The choice
itself is an argmax over these outcomes.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence


def rank_percentile(values: Sequence[float], q: float) -> float:
    """Nearest-rank percentile: the value of rank ceil(q n) (1-based) of the
    sorted values."""
    srt = sorted(values)
    return srt[max(1, math.ceil(q * len(srt))) - 1]


def simulate_worker(robots: int, batch: int, batch_ms: float, t_act_ms: float,
                    n_batches: int) -> Dict[str, float]:
    """One System-1 worker serving ``robots`` closed-loop robots with batch
    size ``batch`` (the reading in the module docstring)."""
    out = {"batch": batch, "feasible": 0, "throughput_hz": 0.0, "action_rate_hz": 0.0,
           "latency_mean_ms": 0.0, "latency_p50_ms": 0.0, "latency_p99_ms": 0.0}
    if robots < batch:
        return out
    out["feasible"] = 1
    pending = [(0.0, r) for r in range(robots)]      # (submission time, robot)
    worker_free = 0.0
    warm = n_batches // 2
    t_warm = 0.0
    latencies: List[float] = []
    for k in range(n_batches):
        pending.sort()
        taken, pending = pending[:batch], pending[batch:]
        start = max(worker_free, taken[-1][0])
        done = start + batch_ms
        for (t_sub, r) in taken:
            if k >= warm:
                latencies.append(done - t_sub)
            pending.append((done + t_act_ms, r))
        worker_free = done
        if k == warm - 1:
            t_warm = done
    span = worker_free - t_warm
    out["throughput_hz"] = len(latencies) * 1000.0 / span
    out["action_rate_hz"] = out["throughput_hz"] / robots
    total = 0.0
    for v in latencies:
        total += v
    out["latency_mean_ms"] = total / len(latencies)
    out["latency_p50_ms"] = rank_percentile(latencies, 0.50)
    out["latency_p99_ms"] = rank_percentile(latencies, 0.99)
    return out


def select_batch(batch_sizes: Sequence[int], batch_ms: Sequence[float], robots: int, t_act_ms: float,
                 slo_ms: float, n_batches: int) -> Optional[int]:
    """Index of the batch size with the highest throughput among those whose
    batches form and whose p99 latency meets the SLO (slo_ms <= 0: none);
    ties go to the smaller batch.  None if no size qualifies."""
    best = None
    for i, (b, t) in enumerate(zip(batch_sizes, batch_ms)):
        o = simulate_worker(robots, b, t, t_act_ms, n_batches)
        if not o["feasible"] or (slo_ms > 0 and o["latency_p99_ms"] > slo_ms):
            continue
        if best is None:
            best = (i, o)
            continue
        bo = best[1]
        if o["throughput_hz"] > bo["throughput_hz"] or \
                (o["throughput_hz"] == bo["throughput_hz"] and b < bo["batch"]):
            best = (i, o)
    return None if best is None else best[0]
