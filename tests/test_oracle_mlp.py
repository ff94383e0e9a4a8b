"""Pins of the oracle's local SGD step (Approach, Eq. 4, second branch)."""
import numpy as np
import pytest
import scipy.special
import torch

import oracle


def _tiny(dims, seed=0, B=3):
    rng = np.random.default_rng(seed)
    params = [(rng.standard_normal((o, i)) * 0.7, rng.standard_normal(o) * 0.3)
              for i, o in zip(dims[:-1], dims[1:])]
    X = rng.standard_normal((B, dims[0]))
    y = rng.integers(0, dims[-1], B)
    return params, X, y


def _loss(params, X, y):
    return oracle.loss_and_grads(params, X, y)[0]


@pytest.mark.parametrize("dims", [(5, 3), (5, 4, 3), (5, 4, 4, 3), (6, 7, 2)])
def test_finite_differences(dims):
    params, X, y = _tiny(dims, seed=len(dims))
    _, grads = oracle.loss_and_grads(params, X, y)
    h = 1e-6
    for l, (W, b) in enumerate(params):
        for arr, g in ((W, grads[l][0]), (b, grads[l][1])):
            num = np.zeros_like(arr)
            for idx in np.ndindex(arr.shape):
                old = arr[idx]
                arr[idx] = old + h
                lp = _loss(params, X, y)
                arr[idx] = old - h
                lm = _loss(params, X, y)
                arr[idx] = old
                num[idx] = (lp - lm) / (2 * h)
            assert np.allclose(g, num, rtol=1e-6, atol=1e-8), (l, g, num)


def test_softmax_regression_closed_form():
    """One layer: grad_W = (P - Y)^T X / B, grad_b = sum_b (P - Y) / B."""
    rng = np.random.default_rng(5)
    B, d, C = 17, 30, 10
    W = rng.standard_normal((C, d)) * 0.1
    b = rng.standard_normal(C) * 0.1
    X = rng.standard_normal((B, d))
    y = rng.integers(0, C, B)
    P = scipy.special.softmax(X @ W.T + b, axis=1)
    Y = np.eye(C)[y]
    loss, grads = oracle.loss_and_grads([(W, b)], X, y)
    assert np.allclose(grads[0][0], (P - Y).T @ X / B, rtol=1e-12, atol=1e-15)
    assert np.allclose(grads[0][1], (P - Y).sum(0) / B, rtol=1e-12, atol=1e-15)
    assert np.isclose(loss, -np.mean(np.log(P[np.arange(B), y])), rtol=1e-12)


def _torch_model(params):
    layers = []
    for l, (W, b) in enumerate(params):
        lin = torch.nn.Linear(W.shape[1], W.shape[0]).double()
        with torch.no_grad():
            lin.weight.copy_(torch.from_numpy(W))
            lin.bias.copy_(torch.from_numpy(b))
        layers.append(lin)
        if l < len(params) - 1:
            layers.append(torch.nn.ReLU())
    return torch.nn.Sequential(*layers)


def test_matches_torch_sgd_step():
    params, X, y = _tiny((12, 9, 7, 4), seed=3, B=8)
    model = _torch_model(params)
    opt = torch.optim.SGD(model.parameters(), lr=0.07)
    loss_t = torch.nn.CrossEntropyLoss()(model(torch.from_numpy(X)), torch.from_numpy(y))
    opt.zero_grad()
    loss_t.backward()
    opt.step()
    new, loss = oracle.sgd_step(params, X, y, 0.07)
    assert np.isclose(loss, loss_t.item(), rtol=1e-13)
    lins = [m for m in model if isinstance(m, torch.nn.Linear)]
    for (W, b), lin in zip(new, lins):
        assert np.allclose(W, lin.weight.detach().numpy(), rtol=1e-12, atol=1e-14)
        assert np.allclose(b, lin.bias.detach().numpy(), rtol=1e-12, atol=1e-14)


def test_bf16_round_matches_torch():
    rng = np.random.default_rng(9)
    x = rng.standard_normal(20000) * np.exp(rng.uniform(-30, 30, 20000))
    # exact ties: float32 values whose low 16 bits are 0x8000, both parities
    ties = (np.arange(1, 200, dtype=np.uint32) << 16 | 0x8000).view(np.float32).astype(np.float64)
    x = np.concatenate([x, ties, -ties, [0.0, -0.0, 1.0, 65504.0, 3.0e38, -3.3e38, np.inf,
                                         -np.inf, np.nan]])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    got = oracle.bf16_round(x)
    assert np.array_equal(got, ref, equal_nan=True)
    fin = ~np.isnan(ref)
    assert np.array_equal(np.signbit(got[fin]), np.signbit(ref[fin]))


def test_bf16_grads_close_to_exact():
    params, X, y = _tiny((40, 32, 24, 10), seed=4, B=16)
    Xq = oracle.bf16_round(X)
    _, g64 = oracle.loss_and_grads(params, Xq, y)
    _, g16 = oracle.loss_and_grads(params, Xq, y, bf16=True)
    for (a, b), (c, d) in zip(g64, g16):
        assert np.linalg.norm(a - c) / np.linalg.norm(a) < 3e-2
        assert np.linalg.norm(b - d) / np.linalg.norm(b) < 3e-2


def test_evaluate_matches_torch():
    """Held-out loss and accuracy: summed CrossEntropyLoss and argmax of an
    nn.Linear / ReLU stack in float64."""
    params, X, y = _tiny((12, 9, 7, 5), seed=8, B=40)
    model = _torch_model(params)
    with torch.no_grad():
        logits = model(torch.from_numpy(X))
        loss_t = torch.nn.CrossEntropyLoss(reduction="sum")(logits, torch.from_numpy(y)).item()
        correct_t = int((logits.argmax(dim=1) == torch.from_numpy(y)).sum())
    loss, correct, gap = oracle.evaluate(params, X, y)
    assert np.isclose(loss, loss_t, rtol=1e-13)
    assert correct == correct_t
    assert gap.shape == (40,) and np.all(gap >= 0.0)


def test_evaluate_counts_ties_and_single_class():
    """A label tied with another class at the top counts as correct; with
    one class every row is correct and the loss is zero."""
    W = np.zeros((3, 2))
    b = np.array([1.0, 1.0, 0.0])
    X = np.ones((4, 2))
    loss, correct, gap = oracle.evaluate([(W, b)], X, [0, 1, 2, 0])
    assert correct == 3 and np.all(gap == 0.0)
    assert np.isclose(loss, 4 * np.log(2 * np.e + 1) - 3 * 1.0)
    loss1, correct1, _ = oracle.evaluate([(np.ones((1, 2)), np.zeros(1))], X, [0, 0, 0, 0])
    assert correct1 == 4 and loss1 == 0.0
