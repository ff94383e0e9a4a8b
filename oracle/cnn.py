"""One local SGD step of a worker on the convolutional workload:
x <- x - eta * g(x) (Approach, Eq. 4, second branch).  The paper trains a
convolutional classifier (ResNet-101 on CIFAR-10, Evaluation Setup); this is
its stand-in for synthetic CIFAR-shaped images.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Readings (the paper fixes no architecture or precision for this build):
* an input row is an image of H x W x C values, channels fastest (NHWC);
* conv layers l = 1..L: 3 x 3 kernels, one zero row and column of padding on
  every side, stride s_l, a bias per output channel, then ReLU:
      Z[b, i, j, o] = bias[o] + sum_{r, s, c} Xpad[b, s_l i + r, s_l j + s, c] W[o, r, s, c]
  for i < H_out = (H - 1) // s_l + 1 (likewise j); W is stored [C_out][3][3][C_in];
* a conv layer l may add the input of the layer before it (A_{l-2}, the
  output of layer l - 2: the input of a two-layer block) to Z before the
  ReLU, the identity shortcut of the residual blocks the paper's ResNet is
  built from: Z_l = conv_l(A_{l-1}) + A_{l-2}; layers l - 1 and l then have
  stride 1 and layer l as many channels as A_{l-2} (l >= 3);
* the mean of every channel over all spatial positions of the last conv layer;
* a fully connected classifier W [classes][C_L] with bias, whose outputs are
  the logits; mean softmax cross-entropy over the batch (as in ``mlp``);
* ReLU'(z) is taken from the stored activation (1 where A > 0);
* every layer's gradient at the same (pre-step) parameters; float64 throughout
  (the paper's PyTorch computes in fp32).

The forward pass is the definition above written out; the backward pass is
the chain rule written out for it (the gradient of a convolution with
respect to its weights correlates the layer's input with the output
gradient; with respect to its input it scatters the output gradient back
through the same kernel taps).

Pinned by tests: the convolution against ``torch.nn.functional.conv2d``
(float64, NCHW), gradients against central finite differences on tiny
networks (with and without a shortcut), and one SGD step against
``torch.optim.SGD`` on an ``nn.Conv2d``/``ReLU``/``AdaptiveAvgPool2d``/
``Linear`` stack with ``CrossEntropyLoss``, with and without shortcuts (CPU,
float64).
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

Params = List[Tuple[np.ndarray, np.ndarray]]


def out_size(n: int, stride: int) -> int:
    """Output extent of a 3 x 3 convolution with padding 1 and this stride."""
    return (n - 1) // stride + 1


def _taps(Xp: np.ndarray, r: int, s: int, stride: int, Ho: int, Wo: int) -> np.ndarray:
    """Xpad[:, stride i + r, stride j + s, :] for all output positions (i, j)."""
    return Xp[:, r:r + stride * (Ho - 1) + 1:stride, s:s + stride * (Wo - 1) + 1:stride, :]


def conv_forward(X: np.ndarray, W: np.ndarray, b: np.ndarray, stride: int) -> np.ndarray:
    """Z of a 3 x 3 convolution, padding 1 (the definition in the module
    docstring).  X [B][H][W][C_in], W [C_out][3][3][C_in] -> [B][Ho][Wo][C_out]."""
    B, H, Wd, _ = X.shape
    Ho, Wo = out_size(H, stride), out_size(Wd, stride)
    Xp = np.pad(X, ((0, 0), (1, 1), (1, 1), (0, 0)))
    Z = np.broadcast_to(np.asarray(b, np.float64), (B, Ho, Wo, W.shape[0])).copy()
    for r in range(3):
        for s in range(3):
            Z += _taps(Xp, r, s, stride, Ho, Wo) @ W[:, r, s, :].T
    return Z


def conv_backward(X: np.ndarray, W: np.ndarray, dZ: np.ndarray, stride: int):
    """Gradients of sum(dZ * conv_forward(X, W, b, stride)) with respect to X,
    W and b."""
    B, H, Wd, C = X.shape
    Ho, Wo, Co = dZ.shape[1], dZ.shape[2], dZ.shape[3]
    Xp = np.pad(X, ((0, 0), (1, 1), (1, 1), (0, 0)))
    dXp = np.zeros_like(Xp)
    dW = np.zeros_like(W)
    flat = dZ.reshape(-1, Co)
    for r in range(3):
        for s in range(3):
            dW[:, r, s, :] = flat.T @ _taps(Xp, r, s, stride, Ho, Wo).reshape(-1, C)
            dXp[:, r:r + stride * (Ho - 1) + 1:stride, s:s + stride * (Wo - 1) + 1:stride, :] += \
                dZ @ W[:, r, s, :]
    return dXp[:, 1:H + 1, 1:Wd + 1, :], dW, flat.sum(axis=0)


def _skips(skips, n: int) -> List[bool]:
    return [bool(v) for v in skips] if skips is not None else [False] * n


def _forward(params: Params, Xb: np.ndarray, image: Sequence[int], strides: Sequence[int],
             skips=None):
    H, Wd, C = image
    acts = [np.asarray(Xb, np.float64).reshape(-1, H, Wd, C)]
    sk = _skips(skips, len(strides))
    for li, ((W, b), st) in enumerate(zip(params[:-1], strides)):
        Z = conv_forward(acts[-1], W, b, st)
        if sk[li]:
            Z = Z + acts[li - 1]  # the input of layer li - 1 (0-based): the block's input
        acts.append(np.maximum(Z, 0.0))
    pooled = acts[-1].mean(axis=(1, 2))
    Wf, bf = params[-1]
    return acts, pooled, pooled @ Wf.T + bf


def loss_and_grads(params: Params, Xb: np.ndarray, yb: Sequence[int], image: Sequence[int],
                   strides: Sequence[int], skips=None):
    """Mean softmax cross-entropy and its gradients at ``params`` = [conv
    layers (W, b) ..., classifier (W, b)].  ``skips``: per conv layer, whether
    it adds its block's input (module docstring).  Returns (loss, grads)."""
    yb = np.asarray(yb, dtype=np.int64)
    acts, pooled, logits = _forward(params, Xb, image, strides, skips)
    sk = _skips(skips, len(strides))
    B = logits.shape[0]
    shift = logits - logits.max(axis=1, keepdims=True)
    expz = np.exp(shift)
    denom = expz.sum(axis=1, keepdims=True)
    loss = float(np.mean(np.log(denom[:, 0]) - shift[np.arange(B), yb]))
    delta = expz / denom
    delta[np.arange(B), yb] -= 1.0
    delta /= B
    Wf = params[-1][0]
    grads: Params = [None] * len(params)
    grads[-1] = (delta.T @ pooled, delta.sum(axis=0))
    A = acts[-1]
    dA = np.broadcast_to((delta @ Wf)[:, None, None, :] / (A.shape[1] * A.shape[2]), A.shape)
    extra = {}  # gradient reaching acts[k] through a shortcut
    for l in range(len(params) - 2, -1, -1):
        if l + 1 in extra:
            dA = dA + extra.pop(l + 1)
        dZ = dA * (acts[l + 1] > 0.0)
        if sk[l]:
            extra[l - 1] = dZ  # Z_l adds acts[l - 1]
        dX, dW, db = conv_backward(acts[l], params[l][0], dZ, strides[l])
        grads[l] = (dW, db)
        dA = dX
    return loss, grads


def sgd_step(params: Params, Xb: np.ndarray, yb: Sequence[int], lr: float,
             image: Sequence[int], strides: Sequence[int], skips=None):
    """x <- x - lr * g(x).  Returns the new parameters and the loss at x."""
    loss, grads = loss_and_grads(params, Xb, yb, image, strides, skips)
    return [(W - lr * dW, b - lr * db) for (W, b), (dW, db) in zip(params, grads)], loss


def evaluate(params: Params, X: np.ndarray, y: Sequence[int], image: Sequence[int],
             strides: Sequence[int], skips=None):
    """Held-out summed softmax cross-entropy and the number of rows whose
    label has the largest logit (ties count), as ``mlp.evaluate``."""
    y = np.asarray(y, dtype=np.int64)
    _, _, logits = _forward(params, X, image, strides, skips)
    n = logits.shape[0]
    top = logits.max(axis=1)
    shift = logits - top[:, None]
    loss_sum = float(np.sum(np.log(np.exp(shift).sum(axis=1)) - shift[np.arange(n), y]))
    return loss_sum, int(np.sum(logits[np.arange(n), y] >= top))
