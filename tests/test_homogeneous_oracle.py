"""Pins of the homogeneous-scheduling oracle (Sec. 3.4.2: obligation
provisioning, binary search on the shared action rate, per-server
configurations from latency profiles, exact packing, closed-loop bound).
No GPU needed."""
import math

import numpy as np
import pytest

from oracle.homogeneous import (ROLE_OBLIGATION, ROLE_S1, ROLE_S2, covers, enumerate_configs, lookup,
                                pack_goal, poisson_arrivals_ms, provision_obligation, rate_profile,
                                schedule_homogeneous, simulate_rate_point, splitmix64)


def test_splitmix64_published_outputs():
    # The reference implementation's first five outputs for seed 1234567.
    want = [6457827717110365317, 3203168211198807973, 9817491932198370423, 4593380528125082431,
            16408922859458223821]
    s, got = 1234567, []
    for _ in range(5):
        s, z = splitmix64(s)
        got.append(z)
    assert got == want


def test_poisson_gaps_are_exponential():
    t = np.array(poisson_arrivals_ms(200.0, 50000, 7))
    gaps = np.diff(np.concatenate([[0.0], t]))
    assert abs(gaps.mean() - 5.0) < 0.05 * 5.0
    # memoryless: P(gap > mean) = e^-1
    assert abs((gaps > 5.0).mean() - math.exp(-1.0)) < 0.01


def test_md1_mean_latency_pollaczek_khinchine():
    # b = 1, service T, Poisson at rho = lambda T: mean sojourn T + rho T / (2 (1 - rho)).
    T = 10.0
    for rho in (0.3, 0.6):
        lam = rho * 1000.0 / T
        mean, _ = simulate_rate_point(1, T, lam, 60000, 3, 0.99)
        want = T + rho * T / (2 * (1 - rho))
        assert abs(mean - want) < 0.03 * want, (rho, mean, want)


def test_light_load_fill_wait():
    # b = 8 at 1% load: the i-th request of a group waits for the b-1-i later
    # ones, on average (b - 1) / (2 lambda), then T.
    b, T = 8, 1.0
    lam = 0.01 * b * 1000.0 / T
    mean, p99 = simulate_rate_point(b, T, lam, 40000, 5, 0.99)
    want = (b - 1) / (2 * lam) * 1000.0 + T
    assert abs(mean - want) < 0.03 * want, (mean, want)
    assert p99 > mean


def test_rate_profile_grid():
    pts = rate_profile(4, 20.0, n_rates=10, n_requests=2000)
    peak = 4 * 1000.0 / 20.0
    assert [round(r, 9) for r, _, _ in pts] == [round(peak * j / 10, 9) for j in range(1, 11)]
    assert all(s >= m for _, m, s in pts)


def test_lookup_reading():
    pts = [(10.0, 5.0, 8.0), (20.0, 7.0, 12.0), (30.0, 11.0, 20.0)]
    assert lookup(pts, 4, 15.0) == (6.0, 10.0)
    assert lookup(pts, 4, 30.0) == (11.0, 20.0)
    assert lookup(pts, 4, 30.5) is None
    assert lookup(pts, 4, 9.0) is None          # fill wait unbounded below the profile
    assert lookup(pts, 1, 9.0) == (5.0, 8.0)    # batch 1: no fill wait
    assert lookup(pts, 4, 10.0) == (5.0, 8.0)


def _const_profile(batch, lat_ms, max_rate):
    return [(batch, [(max_rate * j / 10, lat_ms, lat_ms) for j in range(1, 11)])]


def test_covers_and_obligation_footprint_closed_form():
    # Constant profile up to 100 req/s at 10 req/s per robot: k_max = 10
    # streams per server, so ceil(R / 10) servers.
    m = {"role": ROLE_OBLIGATION, "deadline_ms": 50.0, "profile": _const_profile(1, 5.0, 100.0),
         "rate_per_robot_hz": 10.0}
    for R in (1, 10, 11, 23):
        got = provision_obligation(m, R, 8)
        assert len(got) == math.ceil(R / 10), R
        assert sum(c[1] for c in got) == R
    # memory bound on streams per server
    m2 = dict(m, max_streams=4)
    assert len(provision_obligation(m2, 10, 8)) == 3
    # not enough servers
    assert provision_obligation(m, 23, 2) is None
    cfgs = [(1, 2, 1.0, 1.0), (1, 3, 1.0, 1.0)]
    assert covers(cfgs, 7, 3) == [(0, 0, 1)]         # 2 + 2 + 3
    assert covers(cfgs, 7, 2) == []


def test_pack_prefers_lower_latency_within_budget():
    # Two batch sizes: b=1 serves 2 streams at 10 ms, b=4 serves 4 at 30 ms.
    # 4 robots, budget 2: two b=1 servers (l = 10) beat one b=4 server (l = 30);
    # budget 1: only the b=4 server fits.
    f = 10.0
    m = {"role": ROLE_S1, "deadline_ms": 100.0,
         "profile": _const_profile(1, 10.0, 20.0) + [(4, [(4 * j, 30.0, 30.0) for j in range(1, 11)])]}
    assign, ls = pack_goal([m], f, 4, 2, 1)
    assert ls == [10.0] and sorted(c[0] for c in assign[0]) == [1, 1]
    assign, ls = pack_goal([m], f, 4, 1, 1)
    assert ls == [30.0] and [c[:2] for c in assign[0]] == [(4, 4)]


@pytest.mark.parametrize("R,S,t_act", [(8, 2, 50.0), (8, 8, 50.0), (5, 2, 20.0)])
def test_search_matches_closed_form(R, S, t_act):
    # b = 1 at constant latency T up to lambda_max: a server takes floor(lambda_max / f)
    # streams, so packing holds iff f <= lambda_max / ceil(R / S); the loop bound is
    # 1 / (t_act + T).  The search returns the smaller within eps.
    T, lam = 10.0, 60.0
    m = {"role": ROLE_S1, "deadline_ms": 20.0, "profile": _const_profile(1, T, lam)}
    eps = 1e-4
    out = schedule_homogeneous({"robots": R, "servers": S, "t_act_ms": t_act, "horizon": 1, "eps_hz": eps}, [m])
    want = min(lam / math.ceil(R / S), 1000.0 / (t_act + T))
    assert out["feasible"]
    assert want - 2 * eps <= out["f_hz"] <= want + 1e-12, (out["f_hz"], want)
    assert out["l_s1_ms"] == T
    assert sum(c[1] for _, c in out["assignment"]) == R


def test_obligation_takes_servers_first():
    T, lam = 10.0, 60.0
    s1 = {"role": ROLE_S1, "deadline_ms": 20.0, "profile": _const_profile(1, T, lam)}
    safe = {"role": ROLE_OBLIGATION, "deadline_ms": 20.0, "profile": _const_profile(1, 2.0, 100.0),
            "rate_per_robot_hz": 10.0}
    fleet = {"robots": 12, "servers": 4, "t_act_ms": 10.0, "horizon": 1, "eps_hz": 1e-4}
    out = schedule_homogeneous(fleet, [s1, safe])
    assert out["obligation_servers"] == 2           # 12 robots x 10 Hz at 100 Hz per server
    want = min(lam / math.ceil(12 / 2), 1000.0 / (10.0 + T))
    assert abs(out["f_hz"] - want) <= 2e-4
    alone = schedule_homogeneous(fleet, [s1])
    assert alone["f_hz"] > out["f_hz"]


def test_s2_load_and_latency_are_divided_by_horizon():
    # S2 at constant 200 ms, 40 req/s per server; H = 10 plans reuse.
    T1, T2, H = 10.0, 200.0, 10
    s1 = {"role": ROLE_S1, "deadline_ms": 20.0, "profile": _const_profile(1, T1, 1000.0)}
    s2 = {"role": ROLE_S2, "deadline_ms": 300.0, "profile": _const_profile(1, T2, 40.0)}
    fleet = {"robots": 16, "servers": 2, "t_act_ms": 50.0, "horizon": H, "eps_hz": 1e-4}
    out = schedule_homogeneous(fleet, [s1, s2])
    # one server each; S2 capacity 40 >= 16 f / H up to f = 25; the loop bound binds:
    want = 1000.0 / (50.0 + T1 + T2 / H)
    assert abs(out["f_hz"] - want) <= 2e-4 and out["l_s2_ms"] == T2
    # with H = 1 the S2 capacity binds: 16 f <= 40
    out1 = schedule_homogeneous(dict(fleet, horizon=1), [s1, s2])
    assert abs(out1["f_hz"] - min(40.0 / 16, 1000.0 / (50.0 + T1 + T2))) <= 2e-4


def test_infeasible_deadline():
    m = {"role": ROLE_S1, "deadline_ms": 5.0, "profile": _const_profile(1, 10.0, 60.0)}
    out = schedule_homogeneous({"robots": 2, "servers": 2, "t_act_ms": 50.0, "horizon": 1, "eps_hz": 1e-3}, [m])
    assert not out["feasible"]


def test_enumerate_respects_deadline_and_memory():
    m = {"role": ROLE_S1, "deadline_ms": 25.0, "max_streams": 3,
         "profile": [(1, [(10.0 * j, 5.0 * j, 5.0 * j) for j in range(1, 11)])]}
    got = enumerate_configs(m, 10.0, 8)
    # k streams at 10 Hz each: slo 5 k ms <= 25 and k <= 3
    assert [c[1] for c in got] == [1, 2, 3]
