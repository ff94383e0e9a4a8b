"""Pins of the oracle's convolutional workload (Approach, Eq. 4, second
branch, on the stand-in for the paper's CIFAR-10 convolutional network):
the convolution against torch's conv2d, gradients against central finite
differences, one SGD step and the held-out evaluation against torch modules
(CPU, float64), with and without residual shortcuts."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import cnn


def _net(image, convs, classes, seed, B):
    rng = np.random.default_rng(seed)
    H, W, C = image
    params, cin = [], C
    for co, *_ in convs:
        params.append((rng.standard_normal((co, 3, 3, cin)) * 0.5, rng.standard_normal(co) * 0.2))
        cin = co
    params.append((rng.standard_normal((classes, cin)) * 0.5, rng.standard_normal(classes) * 0.2))
    X = rng.standard_normal((B, H * W * C))
    y = rng.integers(0, classes, B)
    return params, X, y, [c[1] for c in convs]


def _skips(convs):
    return [bool(c[2]) if len(c) > 2 else False for c in convs]


# a residual stack: layer 3 adds the output of layer 1 (the input of its
# two-layer block), layer 6 the output of layer 4
RES = [(4, 1), (5, 1), (4, 1, 1), (6, 2), (3, 1), (6, 1, 1)]


@pytest.mark.parametrize("H,W,C,Co,stride", [(7, 5, 3, 4, 1), (7, 5, 3, 4, 2), (8, 8, 6, 5, 2),
                                             (1, 1, 2, 3, 1), (2, 3, 1, 2, 2)])
def test_conv_matches_torch_conv2d(H, W, C, Co, stride):
    rng = np.random.default_rng(H * 100 + W * 10 + stride)
    X = rng.standard_normal((3, H, W, C))
    Wt = rng.standard_normal((Co, 3, 3, C))
    b = rng.standard_normal(Co)
    got = cnn.conv_forward(X, Wt, b, stride)
    ref = F.conv2d(torch.from_numpy(X).permute(0, 3, 1, 2), torch.from_numpy(Wt).permute(0, 3, 1, 2),
                   torch.from_numpy(b), stride=stride, padding=1).permute(0, 2, 3, 1).numpy()
    assert got.shape == ref.shape
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("convs", [[(4, 1), (3, 2)], [(3, 1), (2, 1), (3, 1, 1)]],
                         ids=["plain", "shortcut"])
def test_finite_differences(convs):
    params, X, y, strides = _net((5, 4, 3), convs, 3, seed=1, B=2)
    img, sk = (5, 4, 3), _skips(convs)
    _, grads = cnn.loss_and_grads(params, X, y, img, strides, sk)
    h = 1e-6
    for l, (Wl, bl) in enumerate(params):
        for arr, g in ((Wl, grads[l][0]), (bl, grads[l][1])):
            num = np.zeros_like(arr)
            for idx in np.ndindex(arr.shape):
                old = arr[idx]
                arr[idx] = old + h
                lp = cnn.loss_and_grads(params, X, y, img, strides, sk)[0]
                arr[idx] = old - h
                lm = cnn.loss_and_grads(params, X, y, img, strides, sk)[0]
                arr[idx] = old
                num[idx] = (lp - lm) / (2 * h)
            assert np.allclose(g, num, rtol=1e-5, atol=1e-8), (l, np.abs(g - num).max())


class _ResidualStack(torch.nn.Module):
    """Conv2d + ReLU layers where a shortcut layer adds the output of the
    layer two before it (its block's input) before its ReLU; then pooling and
    the classifier."""

    def __init__(self, convs, skips, fc):
        super().__init__()
        self.convs = torch.nn.ModuleList(convs)
        self.skips = skips
        self.fc = fc

    def forward(self, x):
        outs = [x]
        for conv, sk in zip(self.convs, self.skips):
            z = conv(outs[-1])
            if sk:
                z = z + outs[-2]
            outs.append(torch.relu(z))
        return self.fc(outs[-1].mean(dim=(2, 3)))


def _torch_model(params, strides, image, skips=None):
    convs, cin = [], image[2]
    for (Wl, bl), st in zip(params[:-1], strides):
        conv = torch.nn.Conv2d(cin, Wl.shape[0], 3, stride=st, padding=1).double()
        with torch.no_grad():
            conv.weight.copy_(torch.from_numpy(Wl).permute(0, 3, 1, 2))
            conv.bias.copy_(torch.from_numpy(bl))
        convs.append(conv)
        cin = Wl.shape[0]
    fc = torch.nn.Linear(cin, params[-1][0].shape[0]).double()
    with torch.no_grad():
        fc.weight.copy_(torch.from_numpy(params[-1][0]))
        fc.bias.copy_(torch.from_numpy(params[-1][1]))
    if skips is None:
        layers = []
        for conv in convs:
            layers += [conv, torch.nn.ReLU()]
        layers += [torch.nn.AdaptiveAvgPool2d(1), torch.nn.Flatten(), fc]
        return torch.nn.Sequential(*layers)
    return _ResidualStack(convs, skips, fc)


def _nchw(X, image):
    H, W, C = image
    return torch.from_numpy(X.reshape(-1, H, W, C)).permute(0, 3, 1, 2).contiguous()


@pytest.mark.parametrize("convs", [[(5, 1), (6, 2), (4, 2)], RES], ids=["plain", "residual"])
def test_matches_torch_sgd_step(convs):
    image = (9, 8, 3)
    params, X, y, strides = _net(image, convs, 4, seed=3, B=5)
    sk = _skips(convs) if any(_skips(convs)) else None
    model = _torch_model(params, strides, image, sk)
    opt = torch.optim.SGD(model.parameters(), lr=0.07)
    loss_t = torch.nn.CrossEntropyLoss()(model(_nchw(X, image)), torch.from_numpy(y))
    opt.zero_grad()
    loss_t.backward()
    opt.step()
    new, loss = cnn.sgd_step(params, X, y, 0.07, image, strides, sk)
    assert np.isclose(loss, loss_t.item(), rtol=1e-13)
    mods = [m for m in model.modules() if isinstance(m, (torch.nn.Conv2d, torch.nn.Linear))]
    for (Wl, bl), m in zip(new, mods):
        w = m.weight.detach()
        if w.dim() == 4:
            w = w.permute(0, 2, 3, 1)
        assert np.allclose(Wl, w.numpy(), rtol=1e-12, atol=1e-14)
        assert np.allclose(bl, m.bias.detach().numpy(), rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("convs", [[(4, 2), (5, 1)], RES], ids=["plain", "residual"])
def test_evaluate_matches_torch(convs):
    image = (6, 6, 3)
    params, X, y, strides = _net(image, convs, 3, seed=4, B=30)
    sk = _skips(convs) if any(_skips(convs)) else None
    model = _torch_model(params, strides, image, sk)
    with torch.no_grad():
        logits = model(_nchw(X, image))
        loss_t = torch.nn.CrossEntropyLoss(reduction="sum")(logits, torch.from_numpy(y)).item()
        correct_t = int((logits.argmax(dim=1) == torch.from_numpy(y)).sum())
    loss, correct = cnn.evaluate(params, X, y, image, strides, sk)
    assert np.isclose(loss, loss_t, rtol=1e-13)
    assert correct == correct_t


def test_rounds_take_the_cnn_step():
    """The oracle's rounds with the convolutional step: K = 1, tau = 1 is one
    SGD step (Eq. 4 reduces to mini-batch SGD)."""
    image = (4, 4, 2)
    params, X, y, strides = _net(image, [(3, 2)], 2, seed=5, B=12)
    step = lambda p, Xb, yb, lr: cnn.sgd_step(p, Xb, yb, lr, image, strides)  # noqa: E731
    res = oracle.run_rounds(params, X, y, 1, np.array([[1]]), 0.1, 4, 99, False, step=step)
    rows = oracle.batch_rows(99, [0, 12], 0, 0, 4)
    ref, _ = cnn.sgd_step(params, X[rows], y[rows], 0.1, image, strides)
    for (a, b), (c, d) in zip(res.params, ref):
        assert np.array_equal(a, c) and np.array_equal(b, d)
