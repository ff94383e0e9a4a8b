"""The load-balancing controller (Approach; Algorithm 1 on measured times) and
the emulated cluster clock (Problem Formulation, Eq. 1), on the host.

The controller's plans are checked against the oracle's quantization and
Algorithm 1 on the same observed times; the barrier and idle time against
Eq. 1 written out on small cases."""
import numpy as np
import pytest

import oracle


@pytest.fixture(scope="module")
def C():
    from paper_2102_08550_amd import controller
    return controller


def test_plans_follow_the_oracle_through_drift_and_jitter(C):
    sched = C.SpeedSchedule([1, 1, 2, 2, 3, 4, 6, 8], {30.0: [8, 6, 4, 3, 2, 2, 1, 1]},
                            jitter=0.03, seed=7)
    lb = C.LoadBalancer(8, M=8, resolution=6)
    base, clock = 1.7, 0.0
    prev_tau = None
    changes = 0
    for r in range(60):
        t = sched.iteration_times(r, clock, base)
        lb.update(t)
        ticks, T, tau = oracle.plan_from_measured(list(t), 6, 8)
        assert (lb.ticks, lb.T_star, lb.tau) == (ticks, T, tau)
        changes += int(prev_tau is not None and tau != prev_tau)
        prev_tau = tau
        clock += C.barrier_time(tau, t)
    assert lb.changes == changes + 1  # the first plan counts as a change
    # after the drift the fastest worker (now worker 0) takes the most steps
    assert lb.tau[0] == max(lb.tau) and lb.tau[-1] == min(lb.tau)


def test_plan_kept_while_ticks_unchanged(C):
    lb = C.LoadBalancer(3, M=8, resolution=4)
    assert lb.update([4.0, 2.0, 1.0]) is True
    assert lb.tau == [1, 2, 4]
    assert lb.update([4.01, 2.02, 1.0]) is False  # same ticks
    assert lb.update([1.0, 2.0, 4.0]) is True and lb.tau == [4, 2, 1]
    assert lb.changes == 2
    with pytest.raises(ValueError):
        lb.update([1.0, 2.0])


def test_barrier_and_idle_time(C):
    # Eq. 1: worker k waits T - tau_k t_k; T = max_k tau_k t_k
    tau, t = [1, 2, 4, 8], [8.0, 4.0, 2.0, 1.0]
    assert C.barrier_time(tau, t) == 8.0 and C.idle_fraction(tau, t) == 0.0
    tau2 = [1, 1, 1, 1]
    assert C.barrier_time(tau2, t) == 8.0
    assert np.isclose(C.idle_fraction(tau2, t), ((8 - 8) + (8 - 4) + (8 - 2) + (8 - 1)) / 32)


def test_schedule_clock_drift_and_jitter(C):
    s = C.SpeedSchedule([1, 2], {5.0: [2, 1]}, jitter=0.1, seed=1)
    assert s.speeds_at(4.99) == [1.0, 2.0] and s.speeds_at(5.0) == [2.0, 1.0]
    a = s.iteration_times(3, 0.0, 2.0)
    assert np.array_equal(a, s.iteration_times(3, 0.0, 2.0))  # same round, same jitter
    assert np.all(np.abs(a / np.array([2.0, 1.0]) - 1.0) <= 0.1)
    b = s.iteration_times(3, 10.0, 2.0)  # after the drift, same jitter draw
    assert np.allclose(b / np.array([1.0, 2.0]), a / np.array([2.0, 1.0]))
    for bad in (dict(speeds=[1, 0]), dict(speeds=[1, 2], changes={1.0: [1]}),
                dict(speeds=[1], jitter=1.0)):
        with pytest.raises(ValueError):
            C.SpeedSchedule(**bad)


def test_fixed_paradigms(C):
    assert C.plan_round("bsp", 3, [1.0, 2.0, 3.0], None, 5) == [1, 1, 1]
    assert C.plan_round("local", 3, [1.0, 2.0, 3.0], None, 5) == [5, 5, 5]
    with pytest.raises(ValueError):
        C.plan_round("asp", 3, [1.0, 2.0, 3.0], None, 5)


def test_batch_schedule(C):
    s = C.BatchSchedule([64, 128, 512, 1024], {3: [1024, 512, 128, 64], 5: [8, 8, 8, 8]})
    assert s.K == 4 and s.max_batch == 1024
    assert s.at(0) == s.at(2) == [64, 128, 512, 1024]
    assert s.at(3) == s.at(4) == [1024, 512, 128, 64]
    assert s.at(9) == [8, 8, 8, 8]
    with pytest.raises(ValueError):
        C.BatchSchedule([64, 0])
    with pytest.raises(ValueError):
        C.BatchSchedule([64, 32], {1: [8]})
