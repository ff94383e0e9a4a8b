"""Writes the expected values of the full-size trajectory tests: the oracle's
run of the two bf16 MLP workloads and the convolutional workloads (plain and
ResNet-style) over all their rounds (Approach, Eq. 4:
every round each worker runs its tau_k local SGD steps from the global model,
then the 1/K average).

    python tests/golden/make_full_size.py [c3] [c5] [c6] [c7]

writes ``tests/golden/full_size_<name>.npz``.  Only ``oracle`` (the
arithmetic) and ``workload`` (the seeded inputs) are called.  A full copy of
the parameters after every round would be hundreds of megabytes, so the file
keeps, per round:
  * ``tau``                    [R][K] local step counts (Algorithm 1 from
                               the speed factors, or the seeded draw);
  * ``loss``                   [R][K] mean training loss of each worker;
  * ``norm_<t>``               [R] L2 norm of tensor t (W1, b1, W2, ...), float64;
  * ``absmax_<t>``             [R] largest magnitude of tensor t;
  * ``idx_<t>``                flat indices kept of tensor t (every element of
                               a tensor of at most FULL elements, else SAMPLE
                               seeded distinct indices, sorted);
  * ``val_<t>``                [len(CHECK)][len(idx)] values at those indices
                               after the rounds in ``check_rounds`` (float32);
  * ``check_rounds``           1-based round numbers kept.
Runtime on 8 cores: about three minutes each (c7: about twenty).
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import workload  # noqa: E402

FULL = 65536
SAMPLE = 8192


def tau_rounds(cfg) -> np.ndarray:
    if cfg.tau_rule == "speeds":
        _, tau = oracle.load_balance(workload.speeds_to_t_iter(cfg.speeds), cfg.M)
        return np.array([tau] * cfg.rounds, dtype=np.int32)
    return workload.gen_tau_uniform(cfg)


def check_rounds(R: int):
    return sorted({1, (R + 1) // 2, R})


def tensor_names(L: int):
    return [f"{kind}{l}" for l in range(1, L + 1) for kind in ("W", "b")]


def make(name: str) -> str:
    cfg = workload.CONFIGS[name]
    t0 = time.time()
    ds = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    X = ds.x_f32().astype(np.float64)
    print(f"{name}: data {X.shape} in {time.time() - t0:.0f} s", flush=True)
    tau = tau_rounds(cfg)
    names = tensor_names(cfg.n_layers)
    shapes = {}
    for l, (W, b) in enumerate(init, start=1):
        shapes[f"W{l}"], shapes[f"b{l}"] = W.shape, b.shape
    rng = np.random.default_rng(20210216)
    idx = {}
    for t in names:
        size = int(np.prod(shapes[t]))
        idx[t] = (np.arange(size, dtype=np.int64) if size <= FULL else
                  np.sort(rng.choice(size, SAMPLE, replace=False)).astype(np.int64))
    checks = check_rounds(cfg.rounds)
    out = {"tau": tau, "check_rounds": np.array(checks, dtype=np.int32),
           "loss": np.zeros((cfg.rounds, cfg.K))}
    for t in names:
        out[f"norm_{t}"] = np.zeros(cfg.rounds)
        out[f"absmax_{t}"] = np.zeros(cfg.rounds)
        out[f"idx_{t}"] = idx[t]
        out[f"val_{t}"] = np.zeros((len(checks), len(idx[t])), dtype=np.float32)
    g = [(W.astype(np.float64), b.astype(np.float64)) for W, b in init]
    steps = None
    seed = workload.sampler_seed(cfg)
    step = None
    if cfg.is_cnn:
        step = lambda p, Xb, yb, lr: oracle.cnn.sgd_step(p, Xb, yb, lr, cfg.image,  # noqa: E731
                                                         cfg.strides, cfg.skips)
    for r in range(cfg.rounds):
        res = oracle.run_rounds(g, X, ds.y, cfg.K, tau[r:r + 1], cfg.lr, cfg.batch, seed,
                                cfg.dtype == workload.BF16, steps_done=steps, step=step)
        g, steps = res.params, res.steps_done
        out["loss"][r] = res.losses[0]
        tensors = {}
        for l, (W, b) in enumerate(g, start=1):
            tensors[f"W{l}"], tensors[f"b{l}"] = W, b
        for t in names:
            flat = tensors[t].ravel()
            out[f"norm_{t}"][r] = np.linalg.norm(flat)
            out[f"absmax_{t}"][r] = np.abs(flat).max()
            if r + 1 in checks:
                out[f"val_{t}"][checks.index(r + 1)] = flat[idx[t]].astype(np.float32)
        print(f"{name}: round {r + 1}/{cfg.rounds} tau={tau[r].tolist()} "
              f"loss={np.round(res.losses[0], 4).tolist()} at {time.time() - t0:.0f} s", flush=True)
    path = os.path.join(HERE, f"full_size_{name}.npz")
    np.savez_compressed(path, **out)
    return path


if __name__ == "__main__":
    for n in (sys.argv[1:] or ["c3", "c5", "c6", "c7"]):
        print("wrote", make(n), flush=True)
