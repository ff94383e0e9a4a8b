"""Round driver over the C ABI.  One Oscars round (Approach, Eq. 4) is either
``oscars_round`` (every worker starts from the global model, runs its tau_k
local SGD steps, and the 1/K average becomes the new global model), or the
two separate calls ``oscars_local_steps`` then ``oscars_aggregate`` with
broadcast (the average written back to every replica).  This module only
moves data into device memory and sequences calls; all arithmetic runs in
the HIP library."""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

from . import BF16, FP32, Context, aggregate, load_balance, paper_weights, shard_offsets


def tau_schedule(cfg, rounds: Optional[int] = None) -> np.ndarray:
    """Per-round local step counts [R][K] of a workload: given, balanced by
    Algorithm 1 from speed factors, or drawn uniformly (an input)."""
    import workload
    R = cfg.rounds if rounds is None else rounds
    if cfg.tau_rule == "given":
        return np.array([cfg.tau_given] * R, dtype=np.int32)
    if cfg.tau_rule == "speeds":
        _, tau = load_balance(workload.speeds_to_t_iter(cfg.speeds), cfg.M)
        return np.array([tau] * R, dtype=np.int32)
    if cfg.tau_rule == "uniform":
        return workload.gen_tau_uniform(cfg)[:R]
    raise ValueError(f"workload {cfg.name} has no local steps")


class OscarsRun:
    """Device state of one workload: dataset, K replicas, global model."""

    def __init__(self, cfg, dataset, init_layers, stream=None):
        import torch
        self.cfg = cfg
        self.dtype = BF16 if cfg.dtype == "bf16" else FP32
        self.ctx = Context(cfg.dims, self.dtype, cfg.K, cfg.batch, stream=stream,
                           cnn=(cfg.image, cfg.conv) if getattr(cfg, "conv", ()) else None)
        dev = torch.device("cuda")
        if self.dtype == BF16:
            self.x = torch.from_numpy(np.ascontiguousarray(dataset.x).view(np.int16)).to(dev)
        else:
            self.x = torch.from_numpy(np.ascontiguousarray(dataset.x)).to(dev)
        self.y = torch.from_numpy(np.ascontiguousarray(dataset.y, dtype=np.int32)).to(dev)
        self.offsets = shard_offsets(dataset.x.shape[0], cfg.K)
        import workload
        self.seed = workload.sampler_seed(cfg)
        flat = torch.from_numpy(self.ctx.pack(init_layers)).to(dev)
        self.n = self.ctx.n_pad
        self.g = flat.clone()
        self.replicas = flat.repeat(cfg.K).contiguous()
        self.weights = paper_weights(cfg.K)

    def local_steps(self, tau: Sequence[int]):
        self.ctx.local_steps(self.replicas, self.x, self.y, self.offsets, self.seed, tau,
                             self.cfg.lr, self.cfg.batch)

    def aggregate(self, broadcast: bool = True):
        aggregate(self.g, self.replicas, self.weights, self.cfg.K, self.n, self.n, broadcast)

    def round(self, tau: Sequence[int]):
        """One round through oscars_round; afterwards ``g`` is the average and
        ``replicas`` the workers' models before averaging."""
        self.ctx.round(self.g, self.replicas, self.x, self.y, self.offsets, self.seed, tau,
                       self.cfg.lr, self.cfg.batch, self.weights)

    def round_broadcast(self, tau: Sequence[int]):
        """The same round as local steps plus aggregation with broadcast."""
        self.local_steps(tau)
        self.aggregate(True)

    def global_layers(self):
        return self.ctx.unpack(self.g.cpu().numpy())

    def close(self):
        self.ctx.close()
