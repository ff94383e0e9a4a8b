"""One local SGD step of a worker: x <- x - eta * g(x) (Approach, Eq. 4,
second branch), for a fully connected ReLU network with a softmax
cross-entropy loss averaged over the mini-batch.

The paper fixes neither the model of the hot path nor the loss; it trains a
classifier (Evaluation Setup) with mini-batch SGD (Related Works, Local SGD).
Readings used:
* layer l computes Z_l = A_{l-1} W_l^T + b_l with W_l stored [out][in];
  hidden layers apply ReLU, the last layer gives the logits;
* loss = mean over the batch of -log softmax(Z_L)[y]; its gradient with
  respect to the logits is (softmax(Z_L) - onehot(y)) / B;
* ReLU'(z) is taken from the stored activation: 1 where A_{l-1} > 0, else 0;
* every layer's gradient is taken at the same (pre-step) parameters.

bf16 workloads (bf16 inputs and weights, fp32 accumulation, fp32 master):
the oracle keeps float64 masters and accumulations and rounds to bf16 at
exactly these points: the weights used by the forward and backward products,
every hidden activation (after ReLU), the logit gradient, and every
propagated gradient (after the ReLU mask).  Inputs are already bf16.  Each
rounding goes float64 -> float32 (round to nearest even) -> bf16 (round to
nearest even on the float32 bits).

Pinned by tests: central finite differences in float64 on tiny networks, the
closed-form gradient of softmax regression, one step of ``torch.optim.SGD``
on ``nn.Linear``/``ReLU``/``CrossEntropyLoss`` (CPU, float64), bf16
rounding against torch's float32 -> bfloat16 conversion, and the bf16
gradient, step and evaluation against an independent torch float64 autograd
reference that rounds at the points listed above (and at no other), with one
negative control per rounding point.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

Params = List[Tuple[np.ndarray, np.ndarray]]


def bf16_round(a: np.ndarray) -> np.ndarray:
    """float64 -> float32 -> bf16 (round to nearest, ties to even), returned as float64.

    On the float32 bit pattern u: add 0x7FFF plus the lowest kept bit, then
    clear the low 16 bits.  Finite patterns are below 0xFF800000, so the sum
    cannot wrap; NaN is kept as NaN and +-inf stay infinite."""
    f = np.asarray(a, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32)
    r = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) & np.uint32(0xFFFF0000)
    out = r.view(np.float32)
    nan = np.isnan(f)
    if nan.any():
        out[nan] = np.nan
    return out.astype(np.float64)


def _identity(a: np.ndarray) -> np.ndarray:
    return a


def loss_and_grads(params: Params, Xb: np.ndarray, yb: Sequence[int], bf16: bool = False):
    """Mean softmax cross-entropy over the batch and its gradients at ``params``.

    Returns (loss, [(dW_1, db_1), ..., (dW_L, db_L)]).
    """
    q = bf16_round if bf16 else _identity
    L = len(params)
    B = Xb.shape[0]
    yb = np.asarray(yb, dtype=np.int64)
    Wq = [q(W) for W, _ in params]
    acts = [np.asarray(Xb, dtype=np.float64)]  # A_0 = the batch
    for l in range(L):
        Z = acts[-1] @ Wq[l].T + params[l][1]
        if l < L - 1:
            acts.append(q(np.maximum(Z, 0.0)))
        else:
            logits = Z
    shift = logits - logits.max(axis=1, keepdims=True)
    expz = np.exp(shift)
    denom = expz.sum(axis=1, keepdims=True)
    loss = float(np.mean(np.log(denom[:, 0]) - shift[np.arange(B), yb]))
    delta = expz / denom
    delta[np.arange(B), yb] -= 1.0
    delta = q(delta / B)
    grads: Params = [None] * L
    for l in range(L - 1, -1, -1):
        dW = delta.T @ acts[l]
        db = delta.sum(axis=0)
        grads[l] = (dW, db)
        if l > 0:
            delta = q((delta @ Wq[l]) * (acts[l] > 0.0))
    return loss, grads


def sgd_step(params: Params, Xb: np.ndarray, yb: Sequence[int], lr: float,
             bf16: bool = False) -> Tuple[Params, float]:
    """x <- x - lr * g(x).  Returns the new parameters and the loss at x."""
    loss, grads = loss_and_grads(params, Xb, yb, bf16)
    new = [(W - lr * dW, b - lr * db) for (W, b), (dW, db) in zip(params, grads)]
    return new, loss


def evaluate(params: Params, X: np.ndarray, y: Sequence[int], bf16: bool = False):
    """Held-out evaluation of a model: the forward pass of ``loss_and_grads``
    (same rounding points) over all rows.  Returns (summed softmax
    cross-entropy, number of rows whose label has the largest logit, and per
    row the gap between the largest and second largest logit, which says
    where float rounding can decide that count)."""
    q = bf16_round if bf16 else _identity
    y = np.asarray(y, dtype=np.int64)
    A = np.asarray(X, dtype=np.float64)
    L = len(params)
    for l, (W, b) in enumerate(params):
        Z = A @ q(W).T + b
        A = q(np.maximum(Z, 0.0)) if l < L - 1 else Z
    logits = A
    n = logits.shape[0]
    top = logits.max(axis=1)
    shift = logits - top[:, None]
    loss_sum = float(np.sum(np.log(np.exp(shift).sum(axis=1)) - shift[np.arange(n), y]))
    correct = int(np.sum(logits[np.arange(n), y] >= top))
    if logits.shape[1] > 1:
        part = np.partition(logits, -2, axis=1)
        gap = part[:, -1] - part[:, -2]
    else:
        gap = np.full(n, np.inf)
    return loss_sum, correct, gap
