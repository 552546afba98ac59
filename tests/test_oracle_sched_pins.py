"""Pins of the scheduler oracle (Section 5.1, Algorithm "Inference") and of the sine
arrival process (Section 7.2): a hand-worked example, closed forms, and the literal
one-microsecond-step loop of the algorithm as brute force."""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import brute
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden():
    g = json.load(open(os.path.join(GOLDEN, "greedy_small.json")))
    return g, {int(k): v for k, v in g["cost"].items()}


def test_greedy_golden_example():
    g, cost = _golden()
    lat, disp = oracle.simulate_greedy(g["arrivals"], g["B"], cost, g["tau"], g["delta"])
    assert [list(d) for d in disp] == g["expected_dispatches"]
    assert lat == g["expected_latency"]
    st = oracle.serving_stats(lat, g["tau"])
    assert st == pytest.approx(g["expected_stats"])


def test_greedy_golden_brute_force():
    g, cost = _golden()
    lat, disp = brute.greedy_busy_loop(g["arrivals"], g["B"], cost, g["tau"], g["delta"], 400)
    assert [list(d) for d in disp] == [d[:2] for d in g["expected_dispatches"]]
    assert lat == g["expected_latency"]


def test_decide_cases():
    B, cost = [16, 32, 48, 64], {16: 70, 32: 120, 48: 180, 64: 230}
    tau, delta = 460, 46
    assert oracle.greedy_decide(B, cost, 64, 0, tau, delta) == 64
    assert oracle.greedy_decide(B, cost, 500, 0, tau, delta) == 64      # never above max(B)
    assert oracle.greedy_decide(B, cost, 15, 10 ** 6, tau, delta) == 0  # below min(B): wait
    assert oracle.greedy_decide(B, cost, 47, 0, tau, delta) == 0
    # largest fitting size, served exactly when c(b) + w + delta reaches tau
    assert oracle.greedy_decide(B, cost, 47, tau - delta - 120 - 1, tau, delta) == 0
    assert oracle.greedy_decide(B, cost, 47, tau - delta - 120, tau, delta) == 32
    assert oracle.greedy_decide(B, cost, 48, tau - delta - 180, tau, delta) == 48


def test_burst_closed_form():
    """k * max(B) requests at t = 0 are served back to back in full batches: batch j
    starts at j c(max B) and its latency is (j + 1) c(max B)."""
    B, cost = [16, 32, 48, 64], {16: 70, 32: 120, 48: 180, 64: 230}
    lat, disp = oracle.simulate_greedy([0] * (5 * 64), B, cost, 460, 46)
    assert disp == [(230 * j, 64, 64 * (5 - j), 230 * j) for j in range(5)]
    assert lat == [230 * (i // 64 + 1) for i in range(5 * 64)]


def test_unit_batch_serves_everything():
    B, cost = [1, 4], {1: 3, 4: 7}
    arr = np.sort(np.random.default_rng(1).integers(0, 500, size=60))
    lat, disp = oracle.simulate_greedy(arr, B, cost, 40, 4)
    assert min(lat) >= 3 and sum(d[1] for d in disp) == 60


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_greedy_matches_literal_loop_on_sine_arrivals(seed):
    """Event-driven oracle == the algorithm's loop stepped every microsecond."""
    B, cost = [16, 32, 48, 64], {16: 700, 32: 1200, 48: 1800, 64: 2300}
    tau = 2 * cost[64]
    arr = wl.sine_arrivals(r_ref=64 / 2300e-6, period_us=100 * tau, duration_us=60_000, step_us=100,
                           seed=seed)
    lat, disp = oracle.simulate_greedy(arr, B, cost, tau, tau // 10)
    lat2, disp2 = brute.greedy_busy_loop(arr, B, cost, tau, tau // 10, 80_000)
    assert len(disp) > 10
    assert [d[:2] for d in disp] == disp2 and lat == lat2


def test_greedy_invariants():
    B, cost = [16, 32, 48, 64], {16: 700, 32: 1200, 48: 1800, 64: 2300}
    tau, delta = 4600, 460
    arr = wl.sine_arrivals(r_ref=64 / 2300e-6, period_us=500 * tau, duration_us=3 * 500 * tau // 2,
                           step_us=460, seed=5)
    lat, disp = oracle.simulate_greedy(arr, B, cost, tau, delta)
    served = sum(d[1] for d in disp)
    assert all(x >= 0 for x in lat[:served]) and all(x == -1 for x in lat[served:])  # FIFO, tail unserved
    assert len(arr) - served < min(B)
    for (t0, b0, q0, w0), (t1, b1, q1, w1) in zip(disp, disp[1:]):
        assert t1 >= t0 + cost[b0]                              # one batch at a time
    for t, b, q, w in disp:
        assert b in B and b <= q
        assert b == max(B) or cost[b] + w + delta >= tau        # the algorithm's two cases
        assert oracle.greedy_decide(B, cost, q, w, tau, delta) == b


def test_sine_rate_shape():
    """Equations (r1)/(r2): the rate exceeds r_ref on 20% of the cycle and peaks at 1.1 r_ref."""
    r_ref, T = 272.0, 1_000_000
    t = np.arange(T)
    r = wl.sine_rate(t, r_ref, T)
    assert r.max() == pytest.approx(1.1 * r_ref, rel=1e-9)
    assert (r >= r_ref).mean() == pytest.approx(0.2, abs=1e-5)
    assert r.min() > 0
    gamma, r0 = wl.sine_coefficients(r_ref)
    assert r.mean() == pytest.approx(r0, rel=1e-9)


def test_sine_arrivals_counts():
    r_ref, T = 500.0, 2_000_000
    arr = wl.sine_arrivals(r_ref, T, 2 * T, 1000, seed=3, noise=0.0)
    gamma, r0 = wl.sine_coefficients(r_ref)
    assert abs(len(arr) - r0 * 2 * T * 1e-6) <= 1          # noise-free: the integral of r
    assert np.all(np.diff(arr) >= 0) and arr.dtype == np.int64
    arr2 = wl.sine_arrivals(r_ref, T, 2 * T, 1000, seed=3)
    assert abs(len(arr2) / len(arr) - 1) < 0.02               # noise has mean zero


# ---------------------------------------------------------------- several servers
def _multi_golden():
    g = json.load(open(os.path.join(GOLDEN, "greedy_multi_small.json")))
    pols = [(p["B"], {int(k): v for k, v in p["cost"].items()}, p["tau"], p["delta"]) for p in g["policies"]]
    return g, pols


def test_greedy_multi_golden_example():
    """Hand-worked two-server example, including a server whose costs fall as b grows
    and that accepts at the same instant after the other server shrank the queue."""
    g, pols = _multi_golden()
    lat, disp = oracle.simulate_greedy_multi(g["arrivals"], pols)
    assert [list(d) for d in disp] == g["expected_dispatches"]
    assert lat == g["expected_latency"]


def test_greedy_multi_golden_brute_force():
    g, pols = _multi_golden()
    lat, disp = brute.greedy_multi_busy_loop(g["arrivals"], pols, 400)
    assert disp == [(d[0], d[1], d[4]) for d in g["expected_dispatches"]]
    assert lat == g["expected_latency"]


def test_greedy_multi_one_server_is_greedy():
    """With one server the shared-queue simulation is the single-model simulation."""
    g, cost = _golden()
    lat, disp = oracle.simulate_greedy_multi(g["arrivals"], [(g["B"], cost, g["tau"], g["delta"])])
    lat1, disp1 = oracle.simulate_greedy(g["arrivals"], g["B"], cost, g["tau"], g["delta"])
    assert lat == lat1 and [d[:4] for d in disp] == [tuple(d) for d in disp1]
    assert all(d[4] == 0 for d in disp)
    B, cost = [16, 32, 48, 64], {16: 700, 32: 1200, 48: 1800, 64: 2300}
    tau = 2 * cost[64]
    for seed in (0, 4):
        arr = wl.sine_arrivals(r_ref=64 / 2300e-6, period_us=100 * tau, duration_us=60_000, step_us=100,
                               seed=seed)
        lat, disp = oracle.simulate_greedy_multi(arr, [(B, cost, tau, tau // 10)])
        lat1, disp1 = oracle.simulate_greedy(arr, B, cost, tau, tau // 10)
        assert len(disp1) > 10
        assert lat == lat1 and [d[:4] for d in disp] == disp1


def _nonmonotone_policies():
    # server 0's batch of 1 costs more than its batch of 2 or 4; server 2 is slow
    return [([1, 2, 4], {1: 460, 2: 150, 4: 210}, 600, 50),
            ([2, 4, 8], {2: 120, 4: 180, 8: 300}, 700, 60),
            ([4], {4: 520}, 900, 80)]


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_greedy_multi_matches_literal_loop(seed):
    """Event-driven multi-server oracle == every server's loop stepped every
    microsecond, on sine arrivals and on random bursts, with non-monotone costs."""
    pols = _nonmonotone_policies()
    if seed < 2:
        arr = wl.sine_arrivals(r_ref=40_000.0, period_us=20_000, duration_us=15_000, step_us=50, seed=seed)
    else:
        rng = np.random.default_rng(seed)
        arr = np.sort(np.concatenate([rng.integers(0, 12_000, size=300), np.full(7, 3000), np.full(5, 9000)]))
    lat, disp = oracle.simulate_greedy_multi(arr, pols)
    lat2, disp2 = brute.greedy_multi_busy_loop(arr, pols, 40_000)
    assert len(disp) > 10 and len({d[4] for d in disp}) == 3
    assert [(d[0], d[1], d[4]) for d in disp] == disp2 and lat == lat2
    starts = [d[0] for d in disp]
    assert starts == sorted(starts)                               # the clock never goes back
    for t, b, q, w, k in disp:
        B, cost, tau, delta = pols[k]
        assert oracle.greedy_decide(B, cost, q, w, tau, delta) == b
