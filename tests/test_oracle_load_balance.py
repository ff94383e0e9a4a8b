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
