"""System-1 batch-size selection: the oracle against closed forms of the
closed-loop worker (Sec. 3.4.2, Step 2.3 bound 1 / (t_act + l_S1); Sec. 4.3,
System-1 batching), then the library's host implementation against the
oracle.  No GPU needed."""
import itertools
import math

import numpy as np
import pytest

from oracle import rank_percentile, select_batch, simulate_worker
from paper_2607_01088_amd import rosa

NB = 240   # the last NB / 2 batches hold whole periods of every regime tested


@pytest.mark.parametrize("b,T,t_act", [(1, 5.0, 0.0), (4, 12.5, 50.0), (16, 30.0, 7.0)])
def test_one_batch_of_robots_cycles_at_t_plus_tact(b, T, t_act):
    o = simulate_worker(b, b, T, t_act, NB)
    assert o["feasible"] == 1
    assert o["latency_p50_ms"] == o["latency_p99_ms"] == T
    assert math.isclose(o["action_rate_hz"], 1000.0 / (T + t_act), rel_tol=1e-12)


@pytest.mark.parametrize("m,b,T", [(2, 4, 10.0), (3, 8, 20.0), (4, 1, 3.0)])
def test_groups_that_never_wait(m, b, T):
    t_act = (m - 1) * T + 1.5          # each group is back after the others' batches
    o = simulate_worker(m * b, b, T, t_act, NB)
    assert math.isclose(o["action_rate_hz"], 1000.0 / (T + t_act), rel_tol=1e-12)
    assert o["latency_p99_ms"] == T


@pytest.mark.parametrize("m,b,T,t_act", [(2, 4, 10.0, 3.0), (4, 16, 20.0, 50.0), (8, 2, 5.0, 0.0)])
def test_saturated_worker_closed_form(m, b, T, t_act):
    assert t_act < (m - 1) * T
    o = simulate_worker(m * b, b, T, t_act, NB)
    assert math.isclose(o["throughput_hz"], 1000.0 * b / T, rel_tol=1e-12)
    assert math.isclose(o["latency_mean_ms"], m * T - t_act, rel_tol=1e-12)


def test_saturated_worker_with_a_partial_group():
    # 3 robots, batches of 2, no action time: the worker never idles, and the
    # leftover robot alternates latencies T and 2T with the others.
    o = simulate_worker(3, 2, 1.0, 0.0, NB)
    assert math.isclose(o["throughput_hz"], 2000.0, rel_tol=1e-12)
    assert (o["latency_p50_ms"], o["latency_p99_ms"], o["latency_mean_ms"]) == (1.0, 2.0, 1.5)


def test_idle_worker_waits_for_the_last_request_of_a_batch():
    # 3 robots, batches of 2, T = 1, t_act = 10: every batch pairs a robot
    # that has waited a whole cycle with one just back, so batches start
    # T + t_act apart and latencies alternate 1 and 12.
    o = simulate_worker(3, 2, 1.0, 10.0, NB)
    assert math.isclose(o["throughput_hz"], 2000.0 / 11.0, rel_tol=1e-12)
    assert (o["latency_p50_ms"], o["latency_p99_ms"], o["latency_mean_ms"]) == (1.0, 12.0, 6.5)


def test_nearest_rank_percentile():
    rng = np.random.default_rng(1)
    for n in [1, 2, 7, 100, 101, 999]:
        v = rng.standard_normal(n)
        for q in [0.01, 0.5, 0.9, 0.99, 1.0]:
            assert rank_percentile(v, q) == np.percentile(v, 100 * q, method="inverted_cdf")


def test_fewer_robots_than_the_batch_is_infeasible():
    o = simulate_worker(3, 4, 1.0, 0.0, NB)
    assert o["feasible"] == 0 and o["throughput_hz"] == 0.0


def test_choice_follows_load_as_the_paper_reports():
    # Sub-linear batch cost (throughput grows with b), as measured for the
    # action expert: light load keeps b = 1, heavy load picks a large batch,
    # an SLO caps the batch.
    sizes = [1, 2, 4, 8, 16, 32]
    ms = [10.0 * b ** 0.5 for b in sizes]
    assert sizes[select_batch(sizes, ms, robots=4, t_act_ms=500.0, slo_ms=0, n_batches=NB)] == 1
    heavy = select_batch(sizes, ms, robots=64, t_act_ms=20.0, slo_ms=0, n_batches=NB)
    assert sizes[heavy] == 32
    # an SLO only admits batch sizes whose p99 latency meets it
    assert sizes[select_batch(sizes, ms, robots=64, t_act_ms=20.0, slo_ms=100.0, n_batches=NB)] == 32
    assert select_batch(sizes, ms, robots=64, t_act_ms=20.0, slo_ms=90.0, n_batches=NB) is None
    assert select_batch([8], [5.0], robots=4, t_act_ms=1.0, slo_ms=0, n_batches=NB) is None


def test_library_simulation_matches_the_oracle():
    for robots, b, T, t_act in itertools.product([1, 3, 16, 50, 256], [1, 2, 5, 16, 64],
                                                 [0.7, 12.5, 61.0], [0.0, 8.0, 200.0]):
        got = rosa.s1_simulate(robots, b, T, t_act, NB)
        ref = simulate_worker(robots, b, T, t_act, NB)
        assert got["feasible"] == ref["feasible"], (robots, b, T, t_act)
        for k in ["throughput_hz", "action_rate_hz", "latency_mean_ms", "latency_p50_ms", "latency_p99_ms"]:
            assert math.isclose(got[k], ref[k], rel_tol=1e-12, abs_tol=1e-12), (k, robots, b, T, t_act)


def test_library_choice_matches_the_oracle():
    rng = np.random.default_rng(0)
    sizes = [1, 2, 4, 8, 16, 32, 64, 128, 256]
    for _ in range(40):
        base = float(rng.uniform(2.0, 20.0))
        expo = float(rng.uniform(0.2, 1.0))
        ms = [base * b ** expo for b in sizes]
        robots = int(rng.integers(1, 300))
        t_act = float(rng.uniform(0.0, 300.0))
        slo = float(rng.choice([0.0, 50.0, 150.0, 400.0]))
        got, outs = rosa.s1_select_batch(sizes, ms, robots, t_act, slo, NB)
        assert got == select_batch(sizes, ms, robots, t_act, slo, NB)
        assert [o["batch"] for o in outs] == sizes


def test_library_rejects_bad_arguments():
    with pytest.raises(rosa.RosaError):
        rosa.s1_simulate(0, 1, 1.0, 0.0)
    with pytest.raises(rosa.RosaError):
        rosa.s1_simulate(4, 1, -1.0, 0.0)
    with pytest.raises(rosa.RosaError):
        rosa.s1_select_batch([2, 2], [1.0, 2.0], 4, 0.0, 0.0)
