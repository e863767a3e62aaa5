"""CPU oracle for homogeneous task scheduling (test infrastructure only).

The paper's steady-state scheduler for a fleet whose robots all run the same
task (Sec. 3.4.2, the homogeneous-scheduling algorithm):

* Step 1: provision each obligation model (safety, monitor) with the fewest
  servers whose measured latency profile meets its deadline under the fleet's
  aggregate load (each robot invokes it at a fixed rate);
* Step 2: binary search the shared action rate f between 0 and f_max, the
  rate with zero inference latency (1 / t_act); for a candidate f every robot
  sends System-1 requests at f and System-2 requests at f / H;
* Step 2.1: the feasible per-server configurations: (model, batch size b, k
  robot streams) whose SLO-percentile latency at the aggregate load (k f or
  k f / H) is within the deadline and whose k fits the server's memory;
* Step 2.2: an exact packing of every goal model's |R| streams onto the
  remaining servers (the paper solves an ILP; here, exhaustive enumeration
  for the tiny instances the tests use);
* Step 2.3: accept f when a packing exists and f <= 1 / (t_act + l_S1 +
  l_S2 / H), l_m the robot-weighted mean latency of model m's chosen servers.

Latency profiles L_m(b, lambda) are tables of (rate, mean, SLO-percentile
latency) points per batch size, ten rates from 10% to 100% of the batch size's
maximum throughput (Sec. 3.4.2, Step 1).  For System 1 they are simulated from
the measured call time T(b) of one batch: Poisson arrivals at the rate (a
SplitMix64 stream, the published generator of Steele, Lea and Flood, turned
into exponential gaps), a batch starts when the server is idle and b requests
wait (the same rule as the batch-size choice), deterministic service T(b).

Readings where the paper is silent:
* a load between two profiled rates takes the linear interpolation of the two
  points; a load above the highest profiled rate is infeasible; a load below
  the lowest profiled rate takes the lowest point only for batch size 1 (no
  fill wait, so latency does not grow as load falls) and is infeasible for
  larger batches (their fill wait grows without bound as load falls);
* the packing's tie-breaking cost (the paper: measured latency and server
  count): minimise l_S1 + l_S2 / H (the closed-loop denominator), then the
  number of servers; obligation footprints minimise servers, then the
  stream-weighted latency;
* the binary search stops when hi - lo <= eps and returns the last accepted f.

Pins (tests marked ``not gpu``): SplitMix64 against its published outputs;
the simulated profile against the M/D/1 Pollaczek-Khinchine mean at b = 1
and the mean fill wait (b - 1) / (2 lambda) at light load; the packing
against the closed form ceil(|R| / k_max) and a hand-solved mixed case; the
search against the closed-form rate of a constant-latency profile (the
closed-loop bound or the capacity bound, whichever binds).
"""
from __future__ import annotations

import itertools
import math
from typing import Dict, List, Optional, Sequence, Tuple

from .s1_batching import rank_percentile

MASK64 = (1 << 64) - 1

ROLE_S1, ROLE_S2, ROLE_OBLIGATION = 0, 1, 2


# ---------------------------------------------------------------- arrivals

def splitmix64(state: int) -> Tuple[int, int]:
    """One step of SplitMix64: (new state, output)."""
    state = (state + 0x9E3779B97F4A7C15) & MASK64
    z = state
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return state, z ^ (z >> 31)


def poisson_arrivals_ms(rate_hz: float, n: int, seed: int) -> List[float]:
    """n arrival times (ms) of a Poisson stream: gap = -ln(u) / rate with
    u = (top 53 bits + 0.5) / 2^53 of successive SplitMix64 outputs."""
    state, t, out = seed & MASK64, 0.0, []
    for _ in range(n):
        state, z = splitmix64(state)
        u = ((z >> 11) + 0.5) / 9007199254740992.0
        t += -math.log(u) * 1000.0 / rate_hz
        out.append(t)
    return out


# ---------------------------------------------------------------- profiles

def simulate_rate_point(batch: int, batch_ms: float, rate_hz: float, n_requests: int, seed: int,
                        pct: float) -> Tuple[float, float]:
    """(mean, pct-percentile) latency in ms of one server with batch size b
    under Poisson arrivals at rate_hz: a batch starts when the server is idle
    and b requests wait, takes the b oldest, returns them after batch_ms.
    Requests of an incomplete last batch are never served and not counted;
    statistics cover the batches after the first tenth."""
    arr = poisson_arrivals_ms(rate_hz, n_requests, seed)
    n_batches = n_requests // batch
    free = 0.0
    lat: List[float] = []
    for j in range(n_batches):
        group = arr[j * batch:(j + 1) * batch]
        start = max(free, group[-1])
        done = start + batch_ms
        free = done
        if j >= n_batches // 10:
            lat.extend(done - t for t in group)
    total = 0.0
    for v in lat:
        total += v
    return total / len(lat), rank_percentile(lat, pct)


def rate_profile(batch: int, batch_ms: float, n_rates: int = 10, n_requests: int = 4000, seed: int = 1,
                 pct: float = 0.99) -> List[Tuple[float, float, float]]:
    """Profile of one batch size: n_rates points (rate, mean, pct latency) at
    j / n_rates of the maximum throughput b / T(b), j = 1 .. n_rates; point j
    uses seed + j."""
    peak = batch * 1000.0 / batch_ms
    pts = []
    for j in range(1, n_rates + 1):
        rate = peak * j / n_rates
        mean, p = simulate_rate_point(batch, batch_ms, rate, n_requests, seed + j, pct)
        pts.append((rate, mean, p))
    return pts


def lookup(points: Sequence[Tuple[float, float, float]], batch: int, load_hz: float
           ) -> Optional[Tuple[float, float]]:
    """(mean, SLO latency) at an aggregate load, from profile points sorted by
    rate (the interpolation reading above), or None if infeasible."""
    if load_hz > points[-1][0]:
        return None
    if load_hz <= points[0][0]:
        if load_hz < points[0][0] and batch != 1:
            return None
        return points[0][1], points[0][2]
    for (r0, m0, s0), (r1, m1, s1) in zip(points[:-1], points[1:]):
        if r0 <= load_hz <= r1:
            w = (load_hz - r0) / (r1 - r0)
            return m0 + w * (m1 - m0), s0 + w * (s1 - s0)
    return None


# ---------------------------------------------------------------- configurations and packing

def enumerate_configs(model: Dict, per_stream_hz: float, robots: int) -> List[Tuple[int, int, float, float]]:
    """Feasible (batch, streams k, mean, slo) for one model at a per-stream
    request rate: k from 1 to min(robots, the model's max_streams)."""
    kmax = robots if not model.get("max_streams") else min(robots, model["max_streams"])
    out = []
    for batch, points in model["profile"]:
        for k in range(1, kmax + 1):
            got = lookup(points, batch, k * per_stream_hz)
            if got is not None and got[1] <= model["deadline_ms"]:
                out.append((batch, k, got[0], got[1]))
    return out


def covers(configs, robots: int, max_servers: int):
    """Every multiset of configurations (as a tuple of indices, non-decreasing)
    whose streams sum to exactly `robots`, with at most max_servers members."""
    res = []

    def rec(start, left, chosen):
        if left == 0:
            res.append(tuple(chosen))
            return
        if len(chosen) == max_servers:
            return
        for i in range(start, len(configs)):
            if configs[i][1] <= left:
                chosen.append(i)
                rec(i, left - configs[i][1], chosen)
                chosen.pop()

    rec(0, robots, [])
    return res


def stream_latency(configs, cover) -> float:
    """Stream-weighted latency sum of a cover: sum of k * mean."""
    s = 0.0
    for i in cover:
        s += configs[i][1] * configs[i][2]
    return s


def provision_obligation(model: Dict, robots: int, servers: int):
    """Fewest servers (then least stream-weighted latency) covering the
    fleet's streams of one obligation model; None if impossible."""
    cfgs = enumerate_configs(model, model["rate_per_robot_hz"], robots)
    best = None
    for cv in covers(cfgs, robots, servers):
        key = (len(cv), stream_latency(cfgs, cv))
        if best is None or key < best[0]:
            best = (key, [cfgs[i] for i in cv])
    return None if best is None else best[1]


def pack_goal(goal_models: Sequence[Dict], f_hz: float, robots: int, budget: int, horizon: int):
    """Exhaustive packing of every goal model's streams within `budget`
    servers, minimising l_S1 + l_S2 / H, then servers.  Returns (assignment
    per model, l per model) or None."""
    per_model = []
    for m in goal_models:
        rate = f_hz if m["role"] == ROLE_S1 else f_hz / horizon
        cfgs = enumerate_configs(m, rate, robots)
        opts = []
        for cv in covers(cfgs, robots, budget):
            opts.append((len(cv), stream_latency(cfgs, cv) / robots, [cfgs[i] for i in cv]))
        if not opts:
            return None
        per_model.append(opts)
    best = None
    for combo in itertools.product(*per_model):
        n = sum(o[0] for o in combo)
        if n > budget:
            continue
        cost = 0.0
        for m, o in zip(goal_models, combo):
            cost += o[1] if m["role"] == ROLE_S1 else o[1] / horizon
        key = (cost, n)
        if best is None or key < best[0]:
            best = (key, combo)
    if best is None:
        return None
    return [o[2] for o in best[1]], [o[1] for o in best[1]]


def schedule_homogeneous(fleet: Dict, models: Sequence[Dict]) -> Dict:
    """The algorithm above.  fleet: robots, servers, t_act_ms, horizon (S2
    plan reuse H), eps_hz.  models: dicts with role, deadline_ms, profile
    [(batch, points)], optional max_streams and (obligations)
    rate_per_robot_hz."""
    R, S = fleet["robots"], fleet["servers"]
    out = {"feasible": False, "f_hz": 0.0, "l_s1_ms": 0.0, "l_s2_ms": 0.0, "obligation_servers": 0,
           "goal_servers": 0, "assignment": []}
    used = 0
    obl = []
    for mi, m in enumerate(models):
        if m["role"] != ROLE_OBLIGATION:
            continue
        got = provision_obligation(m, R, S - used)
        if got is None:
            return out
        used += len(got)
        obl += [(mi, c) for c in got]
    out["obligation_servers"] = used
    budget = S - used
    goal_idx = [i for i, m in enumerate(models) if m["role"] != ROLE_OBLIGATION]
    goal = [models[i] for i in goal_idx]
    H = fleet.get("horizon", 1)
    lo, hi = 0.0, 1000.0 / fleet["t_act_ms"]
    best = None
    while hi - lo > fleet["eps_hz"]:
        f = (lo + hi) / 2
        got = pack_goal(goal, f, R, budget, H)
        ok = False
        if got is not None:
            l1 = sum(l for m, l in zip(goal, got[1]) if m["role"] == ROLE_S1)
            l2 = sum(l for m, l in zip(goal, got[1]) if m["role"] == ROLE_S2)
            f_loop = 1000.0 / (fleet["t_act_ms"] + l1 + l2 / H)
            ok = f <= f_loop
        if ok:
            best = (f, got, l1, l2)
            lo = f
        else:
            hi = f
    if best is None:
        return out
    f, (assign, _), l1, l2 = best
    out.update({"feasible": True, "f_hz": f, "l_s1_ms": l1, "l_s2_ms": l2,
                "goal_servers": sum(len(a) for a in assign),
                "assignment": obl + [(goal_idx[j], c) for j, a in enumerate(assign) for c in a]})
    return out
