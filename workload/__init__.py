"""Seeded synthetic inputs for the Oscars local-SGD hot path.

This module only draws inputs: configurations, Gaussian-mixture data, initial
weights, per-round local step counts, staleness draws and aggregation test
vectors.  It holds none of the method's arithmetic (no load balancing, no
sampling of mini-batches, no forward/backward, no averaging), so both the CPU
oracle and the GPU path may use it without sharing any of the computation.

Recipe (stands in for the paper's CIFAR-10 / ResNet-101 workload, Evaluation
Setup, which is not available here):

* config ``c`` seeds ``numpy.random.SeedSequence(seed)`` and spawns seven
  streams: class means, labels + noise, initial weights, tau draws,
  staleness, aggregation vectors, sampler seed; an eighth stream draws the
  labels and noise of a held-out evaluation set.
* data: C-class Gaussian mixture, mu_c ~ N(0, s^2 I_d) (float32, s =
  ``mean_scale``, 1 unless a workload asks for overlapping classes),
  y ~ U{0..C-1}, x = mu_y + N(0, I_d); bf16 configurations store x rounded
  to bf16 (RNE).
  Rows are drawn in fixed chunks of ``_CHUNK`` rows so that the stream does not
  depend on available memory.
* init: for each layer, W[out][in] then b[out] ~ U(-1/sqrt(in), +1/sqrt(in)),
  float32 (the ``nn.Linear`` convention); convolutional workloads draw each
  conv layer's W[out][3][3][in] and b[out] ~ U(-1/sqrt(9 in), +1/sqrt(9 in))
  (the ``nn.Conv2d`` convention), then the classifier as a linear layer.
* convolutional workloads (the stand-in for the paper's CIFAR-10 images):
  a row is an H x W x C image, channels fastest, drawn from the same mixture.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence, Tuple

import numpy as np

_CHUNK = 8192

FP32 = "fp32"
BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class Config:
    """One workload.  ``dims`` = (d, h_1, ..., C); empty for aggregation-only."""

    name: str
    dims: Tuple[int, ...]
    dtype: str  # "fp32" or "bf16" (bf16 inputs/weights, fp32 accumulation + master)
    K: int  # simulated workers
    n_rows: int  # dataset rows (all workers together)
    batch: int
    tau_rule: str  # "given" | "speeds" | "uniform" | "none"
    tau_given: Tuple[int, ...] = ()
    speeds: Tuple[int, ...] = ()
    tau_range: Tuple[int, int] = (1, 8)
    lr: float = 0.05
    rounds: int = 1
    seed: int = 0
    M: int = 8  # step-difference bound of the barrier constraint
    n_flat: int = 0  # aggregation-only: vector length
    sigma: float = 0.02  # aggregation-only: spread of the replicas around g
    staleness_max: int = 4
    mean_scale: float = 1.0  # class means ~ N(0, mean_scale^2 I): smaller overlaps the classes more
    image: Tuple[int, ...] = ()  # convolutional workloads: (H, W, C) of a row
    # convolutional workloads: (out channels, stride[, shortcut]) per 3x3 layer; a
    # shortcut layer adds the output of the layer two before it (residual block)
    conv: Tuple[Tuple[int, ...], ...] = ()

    @property
    def is_cnn(self) -> bool:
        return bool(self.conv)

    @property
    def n_layers(self) -> int:
        if self.conv:  # conv layers, then the classifier
            return len(self.conv) + 1
        return max(len(self.dims) - 1, 0)

    @property
    def n_classes(self) -> int:
        return self.dims[-1]

    @property
    def d(self) -> int:
        return self.dims[0]

    @property
    def n_params(self) -> int:
        if self.is_cnn:
            n, cin = 0, self.image[2]
            for co, *_ in self.conv:
                n += 9 * cin * co + co
                cin = co
            return n + self.n_classes * cin + self.n_classes
        return sum(o * i + o for i, o in zip(self.dims[:-1], self.dims[1:]))

    @property
    def strides(self) -> Tuple[int, ...]:
        return tuple(c[1] for c in self.conv)

    @property
    def skips(self):
        """Per conv layer, whether it ends a residual block (None: no shortcuts)."""
        sk = tuple(bool(c[2]) if len(c) > 2 else False for c in self.conv)
        return sk if any(sk) else None


# The five workloads the hot path is measured on.  C3/C5 learning rates are not
# given by the workload description; 0.05 (the only MLP value given) is used.
C1 = Config("softmax-reg-784x10-fp32-K4", (784, 10), FP32, K=4, n_rows=8192, batch=32,
            tau_rule="given", tau_given=(1, 2, 3, 4), lr=0.1, rounds=5, seed=1)
C2 = Config("mlp-784-512-256-10-fp32-K8", (784, 512, 256, 10), FP32, K=8, n_rows=60000,
            batch=64, tau_rule="speeds", speeds=(1, 1, 1, 1, 2, 2, 4, 8), lr=0.05,
            rounds=20, seed=2)
C3 = Config("mlp-3072-2048-2048-10-bf16-K16", (3072, 2048, 2048, 10), BF16, K=16,
            n_rows=50000, batch=128, tau_rule="uniform", tau_range=(1, 8), lr=0.05,
            rounds=10, seed=3)
C4 = Config("aggregate-K32-25.6M-fp32", (), FP32, K=32, n_rows=0, batch=0, tau_rule="none",
            rounds=100, seed=4, n_flat=25_600_000, sigma=0.02, staleness_max=4)
C5 = Config("mlp-4096x4-1000-bf16-K8", (4096, 4096, 4096, 4096, 1000), BF16, K=8,
            n_rows=200000, batch=256, tau_rule="speeds", speeds=(1, 1, 2, 2, 3, 4, 6, 8),
            lr=0.05, rounds=5, seed=5)

# Convolutional workload: CIFAR-shaped 32 x 32 x 3 images, 10 classes, three
# 3 x 3 conv layers (32, 64, 128 channels; strides 1, 2, 2), global average
# pooling, a linear classifier; fp32 like the paper's PyTorch; batch 128 as
# in the paper's convergence experiment; 8 workers with the speed factors of
# the 784-512-256-10 workload.
C6 = Config("cnn-32x32x3-c32-c64s2-c128s2-fp32-K8", (3072, 10), FP32, K=8, n_rows=50000,
            batch=128, tau_rule="speeds", speeds=(1, 1, 1, 1, 2, 2, 4, 8), lr=0.05, rounds=5,
            seed=6, image=(32, 32, 3), conv=((32, 1), (64, 2), (128, 2)))

# The same images and workers with a ResNet-style network (the paper's
# ResNet-101 is built of residual blocks): a 32-channel stem, then three stages
# of a conv (stride 1, 2, 2) and a two-layer residual block whose second
# layer adds the stage's first output (identity shortcut), 32 / 64 / 128
# channels.
C7 = Config("cnn-res-32x32x3-c32-r32-c64s2-r64-c128s2-r128-fp32-K8", (3072, 10), FP32, K=8,
            n_rows=50000, batch=128, tau_rule="speeds", speeds=(1, 1, 1, 1, 2, 2, 4, 8), lr=0.05,
            rounds=5, seed=7, image=(32, 32, 3),
            conv=((32, 1), (32, 1), (32, 1, 1), (64, 2), (64, 1), (64, 1, 1), (128, 2), (128, 1),
                  (128, 1, 1)))

CONFIGS = {"c1": C1, "c2": C2, "c3": C3, "c4": C4, "c5": C5, "c6": C6, "c7": C7}


def scaled(cfg: Config, **changes) -> Config:
    """A copy of ``cfg`` with some fields replaced (used for small parity cases)."""
    return dataclasses.replace(cfg, **changes)


def _streams(cfg: Config, count: int = 7):
    # spawn(n)[i] does not depend on n, so the held-out stream (index 7) leaves
    # the first seven unchanged
    ss = np.random.SeedSequence(cfg.seed)
    kids = ss.spawn(count)
    return [np.random.Generator(np.random.PCG64(k)) for k in kids]


def bf16_bits(x32: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round-to-nearest-even) and return the 16-bit
    patterns.  Input storage only: bf16 configurations keep x in this form."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    if not np.all(np.isfinite(x32)):
        raise ValueError("inputs must be finite")
    # finite patterns are at most 0xFF7FFFFF, so the sum stays below 2^32
    r = ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16))
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class Dataset:
    x: np.ndarray  # [n_rows][d] float32, or uint16 bf16 bit patterns
    y: np.ndarray  # [n_rows] int32
    dtype: str

    def x_f32(self) -> np.ndarray:
        return bf16_bits_to_f32(self.x) if self.dtype == BF16 else self.x


def _class_means(cfg: Config, g_means) -> np.ndarray:
    mu = g_means.standard_normal((cfg.n_classes, cfg.d), dtype=np.float32)
    if cfg.mean_scale != 1.0:
        mu *= np.float32(cfg.mean_scale)
    return mu


def _mixture_rows(cfg: Config, mu, g_data, n: int) -> Dataset:
    y = g_data.integers(0, cfg.n_classes, size=n, dtype=np.int64).astype(np.int32)
    out = np.empty((n, cfg.d), dtype=np.uint16 if cfg.dtype == BF16 else np.float32)
    for r0 in range(0, n, _CHUNK):
        r1 = min(n, r0 + _CHUNK)
        blk = g_data.standard_normal((r1 - r0, cfg.d), dtype=np.float32)
        blk += mu[y[r0:r1]]
        out[r0:r1] = bf16_bits(blk) if cfg.dtype == BF16 else blk
    return Dataset(out, y, cfg.dtype)


def gen_eval_set(cfg: Config, n: int) -> Dataset:
    """Held-out rows of the same mixture (same class means, labels and noise
    from a stream of their own), the stand-in for a test set."""
    streams = _streams(cfg, 8)
    return _mixture_rows(cfg, _class_means(cfg, streams[0]), streams[7], n)


def gen_dataset(cfg: Config) -> Dataset:
    """Gaussian mixture: x = mu_y + noise.  bf16 configs store bf16 bit patterns."""
    g_means, g_data = _streams(cfg)[0:2]
    return _mixture_rows(cfg, _class_means(cfg, g_means), g_data, cfg.n_rows)


def gen_init(cfg: Config) -> List[Tuple[np.ndarray, np.ndarray]]:
    """Initial parameters as a list of (W[out][in], b[out]) float32 arrays
    (convolutional workloads: W[out][3][3][in] per conv layer, then the
    classifier's W[classes][channels])."""
    g = _streams(cfg)[2]
    layers = []
    if cfg.is_cnn:
        cin = cfg.image[2]
        for co, *_ in cfg.conv:
            a = 1.0 / math.sqrt(9 * cin)
            W = g.uniform(-a, a, size=(co, 3, 3, cin)).astype(np.float32)
            b = g.uniform(-a, a, size=(co,)).astype(np.float32)
            layers.append((W, b))
            cin = co
        a = 1.0 / math.sqrt(cin)
        layers.append((g.uniform(-a, a, size=(cfg.n_classes, cin)).astype(np.float32),
                       g.uniform(-a, a, size=(cfg.n_classes,)).astype(np.float32)))
        return layers
    for fan_in, fan_out in zip(cfg.dims[:-1], cfg.dims[1:]):
        a = 1.0 / math.sqrt(fan_in)
        W = g.uniform(-a, a, size=(fan_out, fan_in)).astype(np.float32)
        b = g.uniform(-a, a, size=(fan_out,)).astype(np.float32)
        layers.append((W, b))
    return layers


def speeds_to_t_iter(speeds: Sequence[int]) -> np.ndarray:
    """Integer iteration times from relative speeds: t_i = lcm(s) / s_i ticks."""
    L = 1
    for s in speeds:
        L = L * s // math.gcd(L, s)
    return np.array([L // s for s in speeds], dtype=np.int64)


def gen_tau_uniform(cfg: Config) -> np.ndarray:
    """Per-(round, worker) local step counts, integers uniform in tau_range
    (inclusive), for configs whose tau is drawn rather than balanced."""
    g = _streams(cfg)[3]
    lo, hi = cfg.tau_range
    return g.integers(lo, hi + 1, size=(cfg.rounds, cfg.K), dtype=np.int64).astype(np.int32)


def gen_staleness(cfg: Config) -> np.ndarray:
    """Per-(round, worker) staleness, uniform in [0, staleness_max]."""
    g = _streams(cfg)[4]
    return g.integers(0, cfg.staleness_max + 1, size=(cfg.rounds, cfg.K),
                      dtype=np.int64).astype(np.int32)


def gen_agg_vectors(cfg: Config, n: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Aggregation stress inputs: g0 ~ N(0,1) [n] and fixed offsets
    delta_k ~ N(0, sigma^2) [K][n], float32.  Each round's replicas are
    g + delta_k (one float32 add, done identically by every consumer)."""
    g = _streams(cfg)[5]
    n = cfg.n_flat if n is None else n
    g0 = g.standard_normal(n, dtype=np.float32)
    delta = np.empty((cfg.K, n), dtype=np.float32)
    for k in range(cfg.K):
        delta[k] = g.standard_normal(n, dtype=np.float32)
        delta[k] *= np.float32(cfg.sigma)
    return g0, delta


def sampler_seed(cfg: Config) -> int:
    """64-bit seed handed to both samplers."""
    g = _streams(cfg)[6]
    return int(g.integers(0, 2**63 - 1, dtype=np.int64)) * 2 + 1
