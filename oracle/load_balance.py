"""Barrier choice and local step counts (Problem Formulation, Eq. 1-3;
Approach, "Local-SGD load balancing" and Algorithm 1 "Load-Balance").

Pinned by tests against: exhaustive enumeration of the scan window on tiny
integer inputs; the closed form T* = lcm(t) when the lcm lies inside the
window; the speed-factor workloads (tau = speeds); the invariants tau_i >= 1
and "constraint holds at T*".

Readings where the paper is silent or inconsistent:
* times are integer ticks;
* the scan checks the constraint before each candidate T (the for-loop header
  of Algorithm 1), and the history index advances together with T;
* ties in the maximal wait go to the smallest T (indexOf returns the first);
* the scan stops at the first T whose maximal wait is zero: no later T can do
  better and the first-index tie-break would keep it anyway; this is also what
  makes the scan end when all t_i are equal (the constraint then never fails);
* if the constraint already fails at T = max t the problem is infeasible.

Measured iteration times (the controller's input, Problem Formulation: each
worker's iteration time is steady and observed by the global view) are turned
into integer ticks before Algorithm 1: the tick is the fastest worker's time
divided by a resolution R, and each time becomes the nearest whole number of
ticks (halves rounded up), at least one.  The fastest worker is then exactly
R ticks.  Pinned by tests: times that are exact multiples of the tick map to
those multiples, scaling every time by a constant changes nothing, R = 1
gives the fastest worker one tick, and a hand-worked case.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple


class InfeasibleBarrier(ValueError):
    """The barrier constraint fails at the first candidate T = max(t)."""


def wait_times(T: int, t_iter: Sequence[int]) -> List[int]:
    """Eq. 1: idle time of each worker before barrier T, t_i^w = mod(T, t_i)."""
    return [T % int(t) for t in t_iter]


def max_wait(T: int, t_iter: Sequence[int]) -> int:
    """Eq. 2: the largest idle time over all workers."""
    return max(wait_times(T, t_iter))


def barrier_constraint(T: int, t_iter: Sequence[int], M: int) -> bool:
    """Side condition of Eq. 3: floor(T/min t) - floor(T/max t) < M."""
    return T // min(t_iter) - T // max(t_iter) < M


def local_steps_from_barrier(T: int, t_iter: Sequence[int]) -> List[int]:
    """tau_i = floor(T / t_i): iterations worker i completes before T (Eq. 3 text)."""
    return [T // int(t) for t in t_iter]


def load_balance(t_iter: Sequence[int], M: int) -> Tuple[int, List[int]]:
    """Algorithm 1.  Returns (T*, tau).

    Start at T = max t; while the constraint of Eq. 3 holds, record the
    maximal wait (Eq. 2) of T and advance T by one tick; T* is the recorded T
    with the smallest maximal wait.
    """
    t = [int(v) for v in t_iter]
    if not t or min(t) < 1 or M < 1:
        raise ValueError("need at least one worker, t_i >= 1 and M >= 1")
    T = max(t)
    if not barrier_constraint(T, t, M):
        raise InfeasibleBarrier(f"constraint fails at T = max t = {T}")
    max_wait_time: List[int] = []
    T_set: List[int] = []
    while barrier_constraint(T, t, M):
        max_wait_time.append(max_wait(T, t))
        T_set.append(T)
        if max_wait_time[-1] == 0:
            break
        T += 1
    best = min(max_wait_time)
    T_star = T_set[max_wait_time.index(best)]
    return T_star, local_steps_from_barrier(T_star, t)


def quantize_iteration_times(t_measured: Sequence[float], resolution: int) -> List[int]:
    """Measured iteration times (any unit) -> integer ticks, tick = min(t) / R."""
    t = [float(v) for v in t_measured]
    if not t or resolution < 1 or not all(math.isfinite(v) and v > 0.0 for v in t):
        raise ValueError("need positive finite times and a resolution >= 1")
    tick = min(t) / resolution
    return [max(1, int(math.floor(v / tick + 0.5))) for v in t]


def plan_from_measured(t_measured: Sequence[float], resolution: int, M: int):
    """The controller's plan: ticks, then Algorithm 1.  Returns (ticks, T*, tau)."""
    ticks = quantize_iteration_times(t_measured, resolution)
    T_star, tau = load_balance(ticks, M)
    return ticks, T_star, tau
