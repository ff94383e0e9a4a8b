"""Pins of the oracle's Algorithm 1 (Approach, Algorithm 1; Problem
Formulation, Eq. 1-3) against hand-worked cases, exhaustive enumeration, the
lcm closed form and the speed-factor workloads."""
import itertools
import math
import os

import pytest

import oracle
import workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "load_balance.txt")


def _golden_cases():
    out = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        t, M, T, tau = [s.strip() for s in line.split(";")]
        out.append(([int(v) for v in t.split()], int(M), int(T), [int(v) for v in tau.split()]))
    return out


@pytest.mark.parametrize("t,M,T,tau", _golden_cases())
def test_hand_worked(t, M, T, tau):
    assert oracle.load_balance(t, M) == (T, tau)


def _enumerate(t, M, cap=100000):
    """Every T of the scan window [max t, first T violating the constraint),
    evaluated in full, then the first T of least maximal wait."""
    window = []
    T = max(t)
    while T < cap:
        if not (math.floor(T / min(t)) - math.floor(T / max(t)) < M):
            break
        window.append((max(T - ti * math.floor(T / ti) for ti in t), T))
        T += 1
    if not window:
        return None
    best = min(w for w, _ in window)
    return next(T for w, T in window if w == best)


@pytest.mark.parametrize("N", [1, 2, 3])
def test_exhaustive_tiny(N):
    for t in itertools.product(range(1, 7), repeat=N):
        for M in range(1, 7):
            expect = _enumerate(list(t), M)
            if expect is None:
                with pytest.raises(oracle.InfeasibleBarrier):
                    oracle.load_balance(t, M)
                continue
            T, tau = oracle.load_balance(t, M)
            assert T == expect, (t, M)
            assert tau == [T // ti for ti in t]


def test_exhaustive_four_workers_sampled():
    for t in itertools.product((1, 2, 3, 5, 6), repeat=4):
        for M in (2, 5):
            expect = _enumerate(list(t), M)
            if expect is None:
                continue
            assert oracle.load_balance(t, M)[0] == expect


def test_lcm_closed_form():
    """Zero wait happens exactly at multiples of lcm(t); when the lcm lies in
    the scan window it is T*, and every tau_i = lcm / t_i."""
    for t in [(2, 3), (4, 6), (1, 2, 4, 8), (3, 4, 6), (5, 7)]:
        L = math.lcm(*t)
        M = L // min(t) - L // max(t) + 1  # smallest M keeping T = lcm feasible
        T, tau = oracle.load_balance(t, M)
        assert T == L
        assert tau == [L // ti for ti in t]
        assert oracle.max_wait(T, t) == 0


@pytest.mark.parametrize("cfg", [workload.C2, workload.C5])
def test_speed_workloads_give_speeds(cfg):
    t = workload.speeds_to_t_iter(cfg.speeds)
    T, tau = oracle.load_balance(t, cfg.M)
    assert T == math.lcm(*cfg.speeds)
    assert tau == list(cfg.speeds)


def test_invariants_random():
    import random
    rnd = random.Random(7)
    for _ in range(300):
        N = rnd.randint(1, 8)
        t = [rnd.randint(1, 40) for _ in range(N)]
        M = rnd.randint(1, 12)
        try:
            T, tau = oracle.load_balance(t, M)
        except oracle.InfeasibleBarrier:
            assert max(t) // min(t) - 1 >= M
            continue
        assert T >= max(t)
        assert all(x >= 1 for x in tau)
        assert oracle.barrier_constraint(T, t, M)
        assert oracle.wait_times(T, t) == [T - x * ti for x, ti in zip(tau, t)]


def test_infeasible_and_bad_args():
    with pytest.raises(oracle.InfeasibleBarrier):
        oracle.load_balance([1, 10], 5)
    for bad in ([], [0, 1]):
        with pytest.raises(ValueError):
            oracle.load_balance(bad, 3)
    with pytest.raises(ValueError):
        oracle.load_balance([1, 2], 0)


def test_quantize_exact_multiples_and_scale():
    """Times that are whole multiples of the tick give those multiples, at
    any common scale; R = 1 makes the fastest worker one tick."""
    mult = [24, 24, 12, 12, 8, 6, 4, 3]
    for scale in (1.0, 0.37, 1e-3, 2.5e4):
        t = [m * scale for m in mult]
        assert oracle.quantize_iteration_times(t, 3) == mult
        assert oracle.quantize_iteration_times(t, 6) == [2 * m for m in mult]
    assert oracle.quantize_iteration_times([5.0, 10.0, 7.4, 7.6], 1) == [1, 2, 1, 2]


def test_quantize_hand_worked():
    # fastest 2.0 ms, R = 4 -> tick 0.5 ms: 2.0 -> 4, 3.1 -> 6.2 -> 6, 3.25 -> 6.5 -> 7,
    # 9.0 -> 18, 0.26 is never below the fastest; halves round up.
    assert oracle.quantize_iteration_times([2.0, 3.1, 3.25, 9.0], 4) == [4, 6, 7, 18]
    ticks, T, tau = oracle.plan_from_measured([1.0, 2.0, 4.0], 1, 8)
    assert ticks == [1, 2, 4] and T == 4 and tau == [4, 2, 1]


def test_plan_from_measured_noise_robust():
    """Jitter well below half a tick leaves the plan of the speed workload unchanged."""
    rng = __import__("numpy").random.default_rng(3)
    base = [24, 24, 12, 12, 8, 6, 4, 3]
    for _ in range(50):
        t = [b * 1.7 * (1.0 + rng.uniform(-0.01, 0.01)) for b in base]
        ticks, T, tau = oracle.plan_from_measured(t, 3, 8)
        assert ticks == base and T == 24 and tau == [1, 1, 2, 2, 3, 4, 6, 8]


def test_quantize_bad_args():
    for bad in ([], [1.0, 0.0], [1.0, float("nan")], [-1.0]):
        with pytest.raises(ValueError):
            oracle.quantize_iteration_times(bad, 2)
    with pytest.raises(ValueError):
        oracle.quantize_iteration_times([1.0], 0)
