"""Pins of the oracle's bf16 arithmetic: where g(x) of Eq. 4 (Approach) is
rounded to bf16 in the bf16 workloads.

The paper trains in fp32 and fixes no reduced-precision arithmetic, so the
rounding points are a reading: the weights Wq = bf16(W) in both products
(forward and backward-data), every hidden activation after the ReLU, the
logit gradient (softmax - onehot) / B, and every propagated gradient after
the ReLU mask; float64 everywhere else, the masters included.

The pin is an independent implementation of that reading: torch autograd in
float64 on the CPU, where the chain rule is torch's and the rounding enters
only through two custom functions placed at those points -- one that rounds
the value on the way forward (gradient passed through unchanged), one that
rounds the gradient on the way back (value passed through unchanged).  It
must agree with ``oracle.loss_and_grads(bf16=True)`` and
``oracle.evaluate(bf16=True)`` to float64 rounding.  Each rounding point also
has a negative control: the same reference with that one point left out (or
moved) must fail the same comparison, which shows the comparison would catch
an oracle that dropped or moved it."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

REL = 1e-12  # float64 agreement, up to summation order


def _bf16(t: torch.Tensor) -> torch.Tensor:
    # float64 -> float32 (round to nearest even) -> bfloat16 (round to nearest
    # even), torch's own conversions
    return t.to(torch.float32).to(torch.bfloat16).to(torch.float64)


class _RoundValue(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x):
        return _bf16(x)

    @staticmethod
    def backward(ctx, g):
        return g


class _RoundGrad(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x):
        return x.clone()

    @staticmethod
    def backward(ctx, g):
        return _bf16(g)


ALL_POINTS = frozenset({"w_fwd", "w_bwd", "act", "delta_top", "delta_hidden"})


def _torch_reference(params, X, y, points=ALL_POINTS, delta_before_mask=False):
    """Loss and gradients of the mean softmax cross-entropy of a ReLU MLP,
    float64 autograd, bf16 rounding at ``points``:
      w_fwd         weights rounded in the forward product;
      w_bwd         weights rounded in the backward-data product;
      act           hidden activations rounded after the ReLU;
      delta_top     gradient of the logits rounded;
      delta_hidden  gradient of each hidden pre-activation rounded (after the
                    ReLU mask, or before it with ``delta_before_mask``)."""
    Ws = [torch.tensor(W, dtype=torch.float64, requires_grad=True) for W, _ in params]
    bs = [torch.tensor(b, dtype=torch.float64, requires_grad=True) for _, b in params]
    A = torch.tensor(X, dtype=torch.float64)
    L = len(params)
    for l in range(L):
        W = Ws[l]
        if "w_fwd" in points and "w_bwd" in points:
            Wq = _RoundValue.apply(W)
            Z = F.linear(A, Wq, bs[l])
        elif "w_fwd" in points or "w_bwd" in points:
            # one product sees the rounded weights, the other the unrounded ones:
            # Z = A (Wf)^T + b in value, the weight gradient from that term,
            # the input gradient delta Wb from a term that is exactly zero
            Wf = _RoundValue.apply(W) if "w_fwd" in points else W
            Wb = (_bf16(W) if "w_bwd" in points else W).detach()
            Z = F.linear(A.detach(), Wf, bs[l]) + (F.linear(A, Wb) - F.linear(A, Wb).detach())
        else:
            Z = F.linear(A, W, bs[l])
        if l < L - 1:
            if "delta_hidden" in points and not delta_before_mask:
                Z = _RoundGrad.apply(Z)
            H = torch.relu(Z)
            if "delta_hidden" in points and delta_before_mask:
                H = _RoundGrad.apply(H)
            A = _RoundValue.apply(H) if "act" in points else H
        else:
            logits = _RoundGrad.apply(Z) if "delta_top" in points else Z
    loss = F.cross_entropy(logits, torch.tensor(np.asarray(y), dtype=torch.int64))
    loss.backward()
    return loss.item(), [(W.grad.numpy(), b.grad.numpy()) for W, b in zip(Ws, bs)]


def _tiny(dims, seed, B):
    """A tiny network whose every value matters: weights and inputs bf16
    values are not (the masters are float64, inputs bf16 as in the workloads),
    a mix of live and dead ReLUs."""
    rng = np.random.default_rng(seed)
    params = [(rng.standard_normal((o, i)) * (1.3 / np.sqrt(i)), rng.standard_normal(o) * 0.2)
              for i, o in zip(dims[:-1], dims[1:])]
    X = oracle.bf16_round(rng.standard_normal((B, dims[0])))
    y = rng.integers(0, dims[-1], B)
    return params, X, y


def _rel(a, b):
    n = np.linalg.norm(np.asarray(b).ravel())
    return float(np.linalg.norm((np.asarray(a) - np.asarray(b)).ravel()) / max(n, 1e-300))


def _worst(grads_a, grads_b):
    return max(max(_rel(ga, gb), _rel(da, db)) for (ga, da), (gb, db) in zip(grads_a, grads_b))


CASES = [((12, 10, 7), 1, 6), ((16, 24, 20, 5), 2, 9), ((8, 32, 16, 16, 3), 3, 4),
         ((10, 4), 4, 5)]


@pytest.mark.parametrize("dims,seed,B", CASES, ids=[str(c[0]) for c in CASES])
def test_bf16_gradient_matches_torch_reference(dims, seed, B):
    params, X, y = _tiny(dims, seed, B)
    loss, grads = oracle.loss_and_grads(params, X, y, bf16=True)
    loss_t, grads_t = _torch_reference(params, X, y)
    assert abs(loss - loss_t) <= REL * abs(loss_t)
    for l, ((dW, db), (tW, tb)) in enumerate(zip(grads, grads_t)):
        assert _rel(dW, tW) <= REL, (l, _rel(dW, tW))
        assert _rel(db, tb) <= REL, (l, _rel(db, tb))


@pytest.mark.parametrize("dims,seed,B", CASES, ids=[str(c[0]) for c in CASES])
def test_bf16_sgd_step_matches_torch_reference(dims, seed, B):
    """x - lr g(x) with float64 masters: the updated parameters carry no
    rounding of their own."""
    params, X, y = _tiny(dims, seed, B)
    lr = 0.37
    new, _ = oracle.sgd_step(params, X, y, lr, bf16=True)
    _, grads_t = _torch_reference(params, X, y)
    for (W, b), (W0, b0), (tW, tb) in zip(new, params, grads_t):
        assert np.allclose(W, W0 - lr * tW, rtol=0, atol=1e-15 * np.abs(W0).max())
        assert np.allclose(b, b0 - lr * tb, rtol=0, atol=1e-15 * np.abs(b0).max())


CONTROLS = {
    "no weight rounding": dict(points=ALL_POINTS - {"w_fwd", "w_bwd"}),
    "weights unrounded in the forward product": dict(points=ALL_POINTS - {"w_fwd"}),
    "weights unrounded in the backward-data product": dict(points=ALL_POINTS - {"w_bwd"}),
    "hidden activations unrounded": dict(points=ALL_POINTS - {"act"}),
    "logit gradient unrounded": dict(points=ALL_POINTS - {"delta_top"}),
    "propagated gradient unrounded": dict(points=ALL_POINTS - {"delta_hidden"}),
}


@pytest.mark.parametrize("name", list(CONTROLS))
def test_each_rounding_point_is_seen(name):
    """Negative controls: with any one rounding point left out, the torch
    reference no longer agrees with the oracle -- so the comparison above
    pins every point."""
    dims, seed, B = CASES[1]
    params, X, y = _tiny(dims, seed, B)
    _, grads = oracle.loss_and_grads(params, X, y, bf16=True)
    _, grads_c = _torch_reference(params, X, y, **CONTROLS[name])
    assert _worst(grads, grads_c) > 1e3 * REL, name


def test_rounding_after_the_mask_equals_before():
    """Rounding the propagated gradient before or after the ReLU mask is the
    same arithmetic (a masked zero rounds to zero), so that placement needs
    no pin of its own."""
    dims, seed, B = CASES[2]
    params, X, y = _tiny(dims, seed, B)
    _, after = _torch_reference(params, X, y)
    _, before = _torch_reference(params, X, y, delta_before_mask=True)
    assert _worst(after, before) == 0.0


@pytest.mark.parametrize("dims,seed,B", CASES[:3], ids=[str(c[0]) for c in CASES[:3]])
def test_bf16_evaluate_matches_torch_reference(dims, seed, B):
    """Held-out evaluation takes the forward rounding points: summed loss and
    argmax against the torch reference's forward pass; without the weight or
    activation rounding the loss no longer agrees."""
    params, X, y = _tiny(dims, seed, B * 5)
    loss_sum, correct, _ = oracle.evaluate(params, X, y, bf16=True)

    def forward(points):
        A = torch.tensor(X, dtype=torch.float64)
        for l, (W, b) in enumerate(params):
            Wt = torch.tensor(W, dtype=torch.float64)
            Z = F.linear(A, _bf16(Wt) if "w_fwd" in points else Wt,
                         torch.tensor(b, dtype=torch.float64))
            A = (_bf16(torch.relu(Z)) if "act" in points else torch.relu(Z)) \
                if l < len(params) - 1 else Z
        yt = torch.tensor(np.asarray(y), dtype=torch.int64)
        return F.cross_entropy(A, yt, reduction="sum").item(), int((A.argmax(1) == yt).sum())

    ref_loss, ref_correct = forward(ALL_POINTS)
    assert abs(loss_sum - ref_loss) <= REL * abs(ref_loss)
    assert correct == ref_correct
    for drop in ("w_fwd", "act"):
        if drop == "act" and len(params) == 1:
            continue
        other, _ = forward(ALL_POINTS - {drop})
        assert abs(loss_sum - other) > 1e3 * REL * abs(ref_loss), drop
