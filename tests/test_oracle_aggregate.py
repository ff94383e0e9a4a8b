"""Pins of the oracle's aggregation (Approach, Eq. 4: the uniform average)."""
import numpy as np
import pytest

import oracle


@pytest.mark.parametrize("K", [1, 2, 4, 8, 16, 32])
def test_identical_replicas_identity_bitwise(K):
    rng = np.random.default_rng(K)
    x = rng.standard_normal(4097).astype(np.float32)
    g = oracle.tree_aggregate([x.copy() for _ in range(K)], oracle.paper_weights(K))
    assert g.dtype == np.float32
    assert np.array_equal(g.view(np.uint32), x.view(np.uint32))


@pytest.mark.parametrize("K", [3, 5, 7, 12])
def test_identical_replicas_non_power_of_two(K):
    x = np.random.default_rng(K).standard_normal(1000).astype(np.float32)
    g = oracle.tree_aggregate([x] * K, oracle.paper_weights(K))
    assert np.max(np.abs(g - x) / np.abs(x)) < 4 * 2.0**-23


def test_tree_shape_k3_and_k5():
    rng = np.random.default_rng(3)
    xs = [rng.standard_normal(64).astype(np.float32) for _ in range(5)]
    w = [np.float32(v) for v in (0.25, 0.5, 0.125, 0.75, 0.3)]
    l = [w[i] * xs[i] for i in range(5)]
    z = np.zeros(64, np.float32)
    g3 = oracle.tree_aggregate(xs[:3], w[:3])
    assert np.array_equal(g3, (l[0] + l[1]) + (l[2] + z))
    g5 = oracle.tree_aggregate(xs, w)
    assert np.array_equal(g5, ((l[0] + l[1]) + (l[2] + l[3])) + ((l[4] + z) + (z + z)))


def test_float64_reference_random_weights():
    rng = np.random.default_rng(11)
    for K in (2, 6, 32):
        xs = [rng.standard_normal(5000).astype(np.float32) for _ in range(K)]
        w = rng.uniform(0, 1, K).astype(np.float32)
        g = oracle.tree_aggregate(xs, w)
        ref = sum(np.float64(w[k]) * xs[k].astype(np.float64) for k in range(K))
        assert np.linalg.norm(g - ref) / np.linalg.norm(ref) < 1e-6


def test_linearity():
    rng = np.random.default_rng(12)
    K = 8
    g0 = rng.standard_normal(3000).astype(np.float32)
    d = [np.float32(0.02) * rng.standard_normal(3000).astype(np.float32) for _ in range(K)]
    w = oracle.paper_weights(K)
    lhs = oracle.tree_aggregate([g0 + d[k] for k in range(K)], w)
    rhs = g0 + oracle.tree_aggregate(d, w)
    assert np.max(np.abs(lhs - rhs)) < 8 * np.finfo(np.float32).eps * np.max(np.abs(g0))


def test_weights_ignore_staleness():
    for K in (1, 3, 32):
        w0 = oracle.paper_weights(K)
        w1 = oracle.paper_weights(K, staleness=list(range(K)))
        assert np.array_equal(w0, w1)
        assert np.allclose(w0, 1.0 / K)
    with pytest.raises(ValueError):
        oracle.paper_weights(0)
    with pytest.raises(ValueError):
        oracle.paper_weights(3, staleness=[0, 1])


def test_float64_inputs_stay_float64():
    xs = [np.full(3, v, np.float64) for v in (1.0, 2.0, 4.0)]
    g = oracle.tree_aggregate(xs, [1 / 3] * 3)
    assert g.dtype == np.float64
    assert np.allclose(g, 7.0 / 3.0, rtol=1e-15)
