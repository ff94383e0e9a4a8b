"""Pins of the oracle's rounds (Approach, Eq. 4) through the special cases
the method reduces to, plus resume and finiteness on every workload shape."""
import numpy as np
import pytest
import torch

import oracle
import workload


def _setup(dims, K, n_rows, seed):
    cfg = workload.Config("t", tuple(dims), workload.FP32, K=K, n_rows=n_rows, batch=8,
                          tau_rule="given", seed=seed)
    ds = workload.gen_dataset(cfg)
    return cfg, ds.x_f32().astype(np.float64), ds.y, workload.gen_init(cfg)


def _torch_sgd(model, X, y, rows, lr):
    opt = torch.optim.SGD(model.parameters(), lr=lr)
    out = model(torch.from_numpy(X[rows]))
    loss = torch.nn.CrossEntropyLoss()(out, torch.from_numpy(y[rows].astype(np.int64)))
    opt.zero_grad()
    loss.backward()
    opt.step()


def _model(init):
    layers = []
    for l, (W, b) in enumerate(init):
        lin = torch.nn.Linear(W.shape[1], W.shape[0]).double()
        with torch.no_grad():
            lin.weight.copy_(torch.from_numpy(W.astype(np.float64)))
            lin.bias.copy_(torch.from_numpy(b.astype(np.float64)))
        layers.append(lin)
        if l < len(init) - 1:
            layers.append(torch.nn.ReLU())
    return torch.nn.Sequential(*layers)


def _params(model):
    lins = [m for m in model if isinstance(m, torch.nn.Linear)]
    return [(m.weight.detach().numpy(), m.bias.detach().numpy()) for m in lins]


def test_k1_tau1_is_minibatch_sgd():
    cfg, X, y, init = _setup((20, 16, 5), K=1, n_rows=50, seed=21)
    R, lr, B, seed = 12, 0.1, 8, 77
    run = oracle.run_rounds(init, X, y, 1, np.ones((R, 1), int), lr, B, seed, False)
    model = _model(init)
    off = oracle.shard_offsets(len(X), 1)
    for step in range(R):
        _torch_sgd(model, X, y, oracle.batch_rows(seed, off, 0, step, B), lr)
    for (W, b), (Wt, bt) in zip(run.params, _params(model)):
        assert np.allclose(W, Wt, rtol=1e-12, atol=1e-13)
        assert np.allclose(b, bt, rtol=1e-12, atol=1e-13)


def test_equal_tau_is_periodic_model_averaging():
    K, tau, R, lr, B, seed = 4, 3, 4, 0.05, 8, 5
    cfg, X, y, init = _setup((20, 12, 6), K=K, n_rows=120, seed=22)
    run = oracle.run_rounds(init, X, y, K, np.full((R, K), tau), lr, B, seed, False)
    off = oracle.shard_offsets(len(X), K)
    glob = _model(init)
    for r in range(R):
        states = []
        for k in range(K):
            m = _model(_params(glob))
            for j in range(tau):
                _torch_sgd(m, X, y, oracle.batch_rows(seed, off, k, r * tau + j, B), lr)
            states.append(m.state_dict())
        avg = {n: torch.stack([s[n] for s in states]).mean(0) for n in states[0]}
        glob.load_state_dict(avg)
    for (W, b), (Wt, bt) in zip(run.params, _params(glob)):
        assert np.allclose(W, Wt, rtol=1e-11, atol=1e-13)
        assert np.allclose(b, bt, rtol=1e-11, atol=1e-13)


def test_zero_tau_worker_keeps_global():
    cfg, X, y, init = _setup((10, 4), K=3, n_rows=30, seed=23)
    run = oracle.run_rounds(init, X, y, 3, np.array([[2, 0, 1]]), 0.1, 4, 1, False)
    for (W, b), (W0, b0) in zip(run.replicas[1], init):
        assert np.array_equal(W, W0.astype(np.float64)) and np.array_equal(b, b0.astype(np.float64))
    assert run.steps_done == [2, 0, 1]


def test_resume_equals_uninterrupted():
    cfg, X, y, init = _setup((16, 8, 4), K=3, n_rows=45, seed=24)
    tau = np.array([[1, 2, 3], [3, 1, 2], [2, 2, 2], [1, 3, 1]])
    full = oracle.run_rounds(init, X, y, 3, tau, 0.1, 5, 9, False)
    a = oracle.run_rounds(init, X, y, 3, tau[:2], 0.1, 5, 9, False)
    b = oracle.run_rounds(a.params, X, y, 3, tau[2:], 0.1, 5, 9, False, steps_done=a.steps_done)
    assert b.steps_done == full.steps_done
    for (W, bb), (Wf, bf) in zip(b.params, full.params):
        assert np.array_equal(W, Wf) and np.array_equal(bb, bf)


SMALL = {
    "c1": workload.scaled(workload.C1, n_rows=1024, rounds=3),
    "c2": workload.scaled(workload.C2, dims=(784, 64, 32, 10), n_rows=4000, rounds=4),
    "c3": workload.scaled(workload.C3, dims=(3072, 96, 64, 10), n_rows=3200, rounds=3),
    "c5": workload.scaled(workload.C5, dims=(512, 128, 128, 128, 1000), n_rows=8000, rounds=3,
                          batch=64),
}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_workloads_finite_and_learning(name):
    cfg = SMALL[name]
    ds = workload.gen_dataset(cfg)
    if cfg.tau_rule == "given":
        tau = np.array([cfg.tau_given] * cfg.rounds)
    elif cfg.tau_rule == "speeds":
        tau = np.array([oracle.load_balance(workload.speeds_to_t_iter(cfg.speeds), cfg.M)[1]]
                       * cfg.rounds)
    else:
        tau = workload.gen_tau_uniform(cfg)
    run = oracle.run_rounds(workload.gen_init(cfg), ds.x_f32().astype(np.float64), ds.y, cfg.K,
                            tau, cfg.lr, cfg.batch, workload.sampler_seed(cfg),
                            cfg.dtype == workload.BF16)
    losses = [float(np.mean(l)) for l in run.losses]
    assert all(np.isfinite(losses))
    if cfg.n_classes <= 10:
        assert losses[-1] < losses[0]
    else:  # 1000 classes: a few rounds stay on the log(C) plateau; check it does not diverge
        assert max(losses) < np.log(cfg.n_classes) + 0.1
    for W, b in run.params:
        assert np.all(np.isfinite(W)) and np.all(np.isfinite(b))
