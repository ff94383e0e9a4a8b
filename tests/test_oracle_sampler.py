"""Pins of the oracle's shard assignment and mini-batch sampler."""
import collections
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "splitmix64.txt")


def test_splitmix64_published_vectors():
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        seed, outs = line.split(":")
        g = oracle.SplitMix64(int(seed))
        assert [g.next() for _ in outs.split()] == [int(v) for v in outs.split()]


def test_shard_offsets():
    assert oracle.shard_offsets(10, 3) == [0, 3, 6, 10]
    assert oracle.shard_offsets(60000, 8) == [7500 * k for k in range(9)]
    for N, K in [(7, 7), (5, 8), (50000, 16), (200000, 8), (1, 1)]:
        off = oracle.shard_offsets(N, K)
        assert off[0] == 0 and off[-1] == N and len(off) == K + 1
        sizes = np.diff(off)
        assert sizes.min() >= N // K and sizes.max() <= -(-N // K)


def test_each_epoch_is_a_permutation():
    for n in [1, 2, 3, 7, 64, 1000]:
        for k, e in [(0, 0), (3, 1), (15, 7)]:
            p = oracle.epoch_permutation(0x1234, k, e, n)
            assert sorted(p) == list(range(n))


def test_n2_closed_form():
    """For n = 2 the single Fisher-Yates draw j = r mod 2 swaps iff r is even."""
    for seed in range(50):
        for k, e in [(0, 0), (1, 3)]:
            r = oracle.SplitMix64(seed ^ ((k << 32) | e)).next()
            p = oracle.epoch_permutation(seed, k, e, 2)
            assert p == ([1, 0] if r % 2 == 0 else [0, 1])


def test_n3_uniform():
    """All 6 orders of a 3-element shard are (nearly) equally likely."""
    cnt = collections.Counter(tuple(oracle.epoch_permutation(s, 0, 0, 3)) for s in range(6000))
    assert len(cnt) == 6
    chi2 = sum((c - 1000) ** 2 / 1000 for c in cnt.values())
    assert chi2 < 20.5  # p ~ 0.001 at 5 degrees of freedom


def test_batches_cross_epochs_and_persist():
    off = oracle.shard_offsets(23, 4)  # shard sizes 5 6 6 6
    seed = 99
    k = 0
    n_k = off[1] - off[0]
    stream = []
    for step in range(7):  # 7 * 3 = 21 samples = 4 epochs and 1
        stream += oracle.batch_rows(seed, off, k, step, 3)
    for e in range(4):
        assert sorted(stream[e * n_k:(e + 1) * n_k]) == list(range(off[k], off[k + 1]))
        perm = oracle.epoch_permutation(seed, k, e, n_k)
        assert stream[e * n_k:(e + 1) * n_k] == [off[k] + p for p in perm]
    assert stream[20] == off[k] + oracle.epoch_permutation(seed, k, 4, n_k)[0]
    # worker 2's rows stay inside its shard
    rows = oracle.batch_rows(seed, off, 2, 11, 5)
    assert all(off[2] <= r < off[3] for r in rows)


def test_empty_shard_rejected():
    with pytest.raises(ValueError):
        oracle.batch_rows(1, [0, 0, 3], 0, 0, 2)


def test_hand_worked_shuffle():
    path = os.path.join(os.path.dirname(__file__), "golden", "shuffle_n5.txt")
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        head, perm = line.split(":")
        seed, k, e, n = (int(v) for v in head.split())
        assert oracle.epoch_permutation(seed, k, e, n) == [int(v) for v in perm.split()]
