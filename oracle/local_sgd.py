"""Rounds of Oscars local SGD (Approach, Eq. 4).

Reading of Eq. 4 with unequal tau_i: the condition "t mod tau_i = 0" marks
worker i's barrier step.  Every round, each worker starts from the global model
the parameter server broadcast, runs its own tau_i local SGD steps (second
branch), and at the common barrier T* the server averages the N resulting
models uniformly and every worker takes the average (first branch).  Models,
not gradients, are averaged.  Workers are independent between barriers, so
running them one after another gives the same result as running them side by
side.

Full trajectories are "parity unpinned" by the paper (it prints no values);
they are pinned through their parts and through two special cases the tests
check against independent torch loops: K = 1 with tau = 1 is plain mini-batch
SGD, and equal tau with uniform weights is periodic model averaging.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from .aggregate import tree_aggregate
from .mlp import Params, sgd_step
from .sampler import batch_rows, shard_offsets


@dataclasses.dataclass
class OracleRun:
    params: Params  # global model after the last round (float64)
    replicas: List[Params]  # workers' models at the last barrier, before averaging
    steps_done: List[int]  # per-worker step counters
    losses: List[List[float]]  # per round, mean loss of each worker's steps


def worker_local_steps(x0: Params, X: np.ndarray, y: np.ndarray, offsets: Sequence[int],
                       seed: int, k: int, first_step: int, tau: int, lr: float, B: int,
                       bf16: bool, cache: Optional[Dict] = None, step: Optional[Callable] = None):
    """Worker k runs tau SGD steps from x0 on its own shard.  Returns (x, mean
    loss).  ``step(params, Xb, yb, lr) -> (params, loss)`` is the model's SGD
    step (default: the fully connected network of ``mlp``)."""
    x = [(W.copy(), b.copy()) for W, b in x0]
    losses = []
    for j in range(tau):
        rows = batch_rows(seed, offsets, k, first_step + j, B, cache)
        if step is None:
            x, loss = sgd_step(x, X[rows], y[rows], lr, bf16)
        else:
            x, loss = step(x, X[rows], y[rows], lr)
        losses.append(loss)
    return x, (float(np.mean(losses)) if losses else float("nan"))


def _flatten(p: Params) -> List[np.ndarray]:
    out = []
    for W, b in p:
        out += [W, b]
    return out


def run_rounds(init: Params, X: np.ndarray, y: np.ndarray, K: int, tau_rounds: np.ndarray,
               lr: float, B: int, seed: int, bf16: bool, weights: Optional[Sequence[float]] = None,
               steps_done: Optional[Sequence[int]] = None,
               step: Optional[Callable] = None) -> OracleRun:
    """Run ``len(tau_rounds)`` rounds; ``tau_rounds[r][k]`` is worker k's step
    count in round r.  ``X`` holds the inputs as float64 (bf16 values for bf16
    workloads), ``init`` the starting global model, ``step`` the model's SGD
    step (see worker_local_steps)."""
    offsets = shard_offsets(X.shape[0], K)
    g = [(np.asarray(W, np.float64).copy(), np.asarray(b, np.float64).copy()) for W, b in init]
    w = np.full(K, 1.0 / K) if weights is None else np.asarray(weights, np.float64)
    s = list(steps_done) if steps_done is not None else [0] * K
    cache: Dict = {}
    losses = []
    replicas: List[Params] = []
    for tau in tau_rounds:
        replicas, round_losses = [], []
        for k in range(K):
            xk, lk = worker_local_steps(g, X, y, offsets, seed, k, s[k], int(tau[k]), lr, B,
                                        bf16, cache, step)
            replicas.append(xk)
            round_losses.append(lk)
            s[k] += int(tau[k])
        flat = [_flatten(r) for r in replicas]
        new = [tree_aggregate([flat[k][i] for k in range(K)], w) for i in range(len(flat[0]))]
        g = [(new[2 * l], new[2 * l + 1]) for l in range(len(g))]
        losses.append(round_losses)
    return OracleRun(g, replicas, s, losses)
