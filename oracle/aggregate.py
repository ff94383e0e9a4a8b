"""Parameter-server aggregation (Approach, Eq. 4, first branch: the average
(1/N) sum_k of the workers' models at the barrier).

Reading: the paper's weight is uniform, w_k = 1/N, independent of tau_k and of
any staleness (no other weighting is defined).  The summation order, which the
paper leaves open, is a balanced pairwise tree: with P the next power of two
>= K, leaf k is fl(w_k * x_k) for k < K and +0 otherwise; each inner node is
fl(left + right), level by level.  Floating-point addition is commutative, so
only this grouping matters.

Pinned by tests: identical replicas give the identity (bit for bit when K is a
power of two); linearity; agreement with a float64 sum for random non-uniform
weights; a K = 3 tree written out by hand.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np


def paper_weights(K: int, staleness: Optional[Sequence[int]] = None) -> np.ndarray:
    """Eq. 4 weights w_k = 1/K as float32.  ``staleness`` is accepted and has
    no effect: the update rule averages uniformly."""
    if K < 1:
        raise ValueError("K >= 1 required")
    if staleness is not None and len(staleness) != K:
        raise ValueError("one staleness value per worker")
    return np.full(K, np.float32(1.0) / np.float32(K), dtype=np.float32)


def tree_aggregate(replicas: Sequence[np.ndarray], weights: Sequence[float]) -> np.ndarray:
    """g = pairwise-tree sum of w_k * x_k, evaluated in the replicas' dtype."""
    K = len(replicas)
    if K < 1 or len(weights) != K:
        raise ValueError("one weight per replica")
    dt = np.asarray(replicas[0]).dtype
    P = 1
    while P < K:
        P *= 2
    level = []
    for k in range(P):
        if k < K:
            level.append(dt.type(weights[k]) * np.asarray(replicas[k], dtype=dt))
        else:
            level.append(np.zeros_like(np.asarray(replicas[0], dtype=dt)))
    while len(level) > 1:
        level = [level[i] + level[i + 1] for i in range(0, len(level), 2)]
    return level[0]
