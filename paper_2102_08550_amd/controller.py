"""Global-view load balancing and the comparison of synchronization paradigms.

The load balancer is the controller of the Approach: it observes every
worker's iteration time t_i^iter (Problem Formulation: steady per worker,
different across a heterogeneous cluster), turns the times into integer ticks
and runs Algorithm 1 (``oscars_plan_tau``), and re-plans whenever the
quantized times change.  Slower workers then take fewer local steps between
two averagings and faster workers more (Motivation, Figure "Local SGD with
load-balancing").

The heterogeneous cluster is emulated: worker k runs at a relative speed s_k
(which may change from a given clock time on), and its iteration time is a
measured GPU step time divided by s_k, times a seeded jitter factor.  All
workers' arithmetic runs on this GPU through ``oscars_round``; only the clock
of the cluster is modelled.  A round ends at the barrier of Eq. 1, when the
last worker finishes: max_k tau_k t_k.  As in Problem Formulation, the time
of the parameter exchange itself is not counted.

``run_measured`` closes the loop on measured times instead: the workers'
work differs for real (each worker draws its own mini-batch size, which Eq. 4
leaves free), every worker's local steps run as launches of their own, and
its iteration time is the GPU time of those launches (HIP events around each
launch, summed) divided by its step count.  The load balancer plans the next
round from these measurements, so a change in a worker's work is followed by
a new plan.

Paradigms compared (Motivation):
  * ``bsp``    -- synchronous mini-batch SGD by averaging: tau_k = 1;
  * ``local``  -- local SGD without balancing: tau_k = I for every worker;
  * ``oscars`` -- local SGD with the load balancer's tau.

Run as ``python -m paper_2102_08550_amd.controller`` for the comparison on the
784-512-256-10 MLP workload (8 workers with speeds 1,1,1,1,2,2,4,8 that
drift half way); it prints one JSON object.
"""
from __future__ import annotations

import argparse
import json
import sys
import time
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import plan_tau

PARADIGMS = ("bsp", "local", "oscars")


class SpeedSchedule:
    """Relative worker speeds over the emulated clock, with optional drift
    and jitter.

    ``changes`` maps a clock time, in units of the speed-1 iteration time, to
    the speeds used from then on, so every paradigm meets the drift at the
    same time.  The iteration time of worker k in a round that starts at
    clock c is base / s_k(c) * (1 + u), u uniform in [-jitter, jitter] from a
    generator seeded by (seed, round), identical for every paradigm."""

    def __init__(self, speeds: Sequence[float], changes: Optional[Dict[int, Sequence[float]]] = None,
                 jitter: float = 0.0, seed: int = 0):
        self.speeds = [float(s) for s in speeds]
        self.changes = {float(c): [float(s) for s in v] for c, v in (changes or {}).items()}
        if any(s <= 0 for s in self.speeds) or any(s <= 0 for v in self.changes.values() for s in v):
            raise ValueError("speeds must be positive")
        if any(len(v) != len(self.speeds) for v in self.changes.values()):
            raise ValueError("every speed vector needs one speed per worker")
        if not 0.0 <= jitter < 1.0:
            raise ValueError("jitter must be in [0, 1)")
        self.jitter = float(jitter)
        self.seed = int(seed)

    @property
    def K(self) -> int:
        return len(self.speeds)

    def speeds_at(self, clock_units: float) -> List[float]:
        cur = self.speeds
        for start in sorted(self.changes):
            if start <= clock_units:
                cur = self.changes[start]
        return list(cur)

    def iteration_times(self, r: int, clock: float, base: float) -> np.ndarray:
        """Worker iteration times of round r (r >= -1; -1 is the measurement
        before training), which starts at ``clock`` (same unit as ``base``,
        the speed-1 iteration time)."""
        if r < -1:
            raise ValueError("round index below -1")
        s = np.asarray(self.speeds_at(clock / base), dtype=np.float64)
        t = base / s
        if self.jitter > 0.0:
            g = np.random.default_rng([self.seed, r + 1])  # r = -1: before training
            t = t * (1.0 + g.uniform(-self.jitter, self.jitter, size=len(s)))
        return t


class LoadBalancer:
    """The global-view controller: plan tau from measured iteration times.
    A new plan (ticks, T*, tau) is adopted when the quantized times change;
    ``changes`` counts the plans whose tau differs from the previous one."""

    def __init__(self, K: int, M: int = 8, resolution: int = 8):
        self.K, self.M, self.resolution = int(K), int(M), int(resolution)
        self.ticks: Optional[List[int]] = None
        self.T_star: Optional[int] = None
        self.tau: Optional[List[int]] = None
        self.changes = 0

    def update(self, t_measured: Sequence[float]) -> bool:
        """Feed one measurement of every worker's iteration time; returns True
        when tau changed."""
        if len(t_measured) != self.K:
            raise ValueError("one time per worker")
        ticks, T, tau = plan_tau(t_measured, self.resolution, self.M)
        if ticks == self.ticks:
            return False
        changed = tau != self.tau
        self.ticks, self.T_star, self.tau = ticks, T, tau
        self.changes += int(changed)
        return changed


def barrier_time(tau: Sequence[int], t_iter: Sequence[float]) -> float:
    """Eq. 1: the round ends when the last worker finishes its tau_k steps."""
    return float(max(int(a) * float(t) for a, t in zip(tau, t_iter)))


def idle_fraction(tau: Sequence[int], t_iter: Sequence[float]) -> float:
    """Share of worker time spent waiting at the barrier (sum of t_k^w over K T)."""
    T = barrier_time(tau, t_iter)
    busy = sum(int(a) * float(t) for a, t in zip(tau, t_iter))
    return 1.0 - busy / (len(tau) * T) if T > 0 else 0.0


def plan_round(paradigm: str, K: int, observed: Sequence[float],
               balancer: Optional[LoadBalancer], local_steps: int) -> List[int]:
    """tau of the next round.  The load balancer plans from the iteration
    times observed in the previous round (before the first round: one
    measurement of every worker)."""
    if paradigm == "bsp":
        return [1] * K
    if paradigm == "local":
        return [int(local_steps)] * K
    if paradigm == "oscars":
        balancer.update(observed)
        return list(balancer.tau)
    raise ValueError(f"unknown paradigm {paradigm!r}")


def measure_step_ms(cfg, dataset, init, reps: int = 5) -> float:
    """GPU time of one local step of one worker (median of ``reps``), on a
    context of its own: the iteration time of a speed-1 worker."""
    import torch

    from .rounds import OscarsRun
    run = OscarsRun(cfg, dataset, init)
    try:
        tau = [1] + [0] * (cfg.K - 1)
        for _ in range(2):
            run.local_steps(tau)
        times = []
        for _ in range(reps):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            run.local_steps(tau)
            b.record()
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b))
    finally:
        run.close()
    return float(np.median(times))


def run_paradigm(cfg, dataset, init, eval_set, paradigm: str, schedule: SpeedSchedule,
                 base: float, time_budget: float, local_steps: int = 4, resolution: int = 8,
                 max_rounds: int = 100000, eval_every: int = 1,
                 return_model: bool = False) -> Dict:
    """Train with one paradigm until the emulated cluster clock reaches
    ``time_budget`` (same unit as ``base``).  Returns per-round records (and
    the final global model as layers when ``return_model``)."""
    import torch

    from .rounds import OscarsRun
    K = cfg.K
    if schedule.K != K:
        raise ValueError("schedule and workload disagree on K")
    balancer = LoadBalancer(K, cfg.M, resolution) if paradigm == "oscars" else None
    run = OscarsRun(cfg, dataset, init)
    dev = torch.device("cuda")
    xe = np.ascontiguousarray(eval_set.x)
    x_eval = torch.from_numpy(xe.view(np.int16) if xe.dtype == np.uint16 else xe).to(dev)
    y_eval = torch.from_numpy(np.ascontiguousarray(eval_set.y, dtype=np.int32)).to(dev)
    n_eval = int(y_eval.shape[0])
    records = []
    clock = 0.0
    samples = 0
    gpu_ms = 0.0
    try:
        loss0, hit0 = run.ctx.evaluate(run.g, x_eval, y_eval)
        records.append({"round": -1, "clock": 0.0, "samples": 0, "eval_loss": loss0 / n_eval,
                        "eval_acc": hit0 / n_eval})
        r = 0
        observed = schedule.iteration_times(-1, 0.0, base)
        while clock < time_budget and r < max_rounds:
            tau = plan_round(paradigm, K, observed, balancer, local_steps)
            t_true = schedule.iteration_times(r, clock, base)
            observed = t_true
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            run.round(tau)
            b.record()
            torch.cuda.synchronize()
            gpu_ms += a.elapsed_time(b)
            clock += barrier_time(tau, t_true)
            samples += int(sum(tau)) * cfg.batch
            rec = {"round": r, "clock": clock, "samples": samples, "tau": list(tau),
                   "idle": idle_fraction(tau, t_true)}
            if balancer is not None:
                rec["T_star"] = balancer.T_star
                rec["ticks"] = list(balancer.ticks)
            if (r + 1) % eval_every == 0:
                loss, hit = run.ctx.evaluate(run.g, x_eval, y_eval)
                rec["eval_loss"] = loss / n_eval
                rec["eval_acc"] = hit / n_eval
            records.append(rec)
            r += 1
        model = run.global_layers() if return_model else None
    finally:
        run.close()
    return {"paradigm": paradigm, "records": records, "model": model, "gpu_ms": gpu_ms, "samples": samples,
            "tau_changes": balancer.changes if balancer else 0}


class BatchSchedule:
    """Per-worker mini-batch sizes over the rounds: ``batches`` from round 0
    on, replaced by ``changes[r]`` from round r on.  A worker whose batch
    size changes continues its sample stream at step position cursor x new
    size (Eq. 4 fixes no mini-batch rule; the oracle reads positions the same
    way)."""

    def __init__(self, batches: Sequence[int], changes: Optional[Dict[int, Sequence[int]]] = None):
        self.batches = [int(b) for b in batches]
        self.changes = {int(r): [int(b) for b in v] for r, v in (changes or {}).items()}
        if any(b < 1 for b in self.batches) or any(b < 1 for v in self.changes.values() for b in v):
            raise ValueError("batch sizes must be positive")
        if any(len(v) != len(self.batches) for v in self.changes.values()):
            raise ValueError("one batch size per worker")

    @property
    def K(self) -> int:
        return len(self.batches)

    @property
    def max_batch(self) -> int:
        return max([max(self.batches)] + [max(v) for v in self.changes.values()])

    def at(self, r: int) -> List[int]:
        cur = self.batches
        for start in sorted(self.changes):
            if start <= r:
                cur = self.changes[start]
        return list(cur)


def run_measured(cfg, dataset, init, schedule: BatchSchedule, rounds: int, resolution: int = 4,
                 return_model: bool = False) -> Dict:
    """Oscars with the load balancer fed by measured iteration times.

    Round 0 is a probe: every worker takes one step.  In every round worker k
    runs its tau_k local steps with its own mini-batch size as launches of its
    own (``oscars_local_steps`` with only worker k active; the result equals
    the grouped launches bit for bit), HIP events around each of those
    launches give its GPU time, and t_k = that time / tau_k.  Then the
    parameter server averages and broadcasts (``oscars_aggregate``).  The
    next round's tau is Algorithm 1 on the ticks of the measured t
    (``LoadBalancer``).  Returns per-round records: tau, batch sizes,
    measured times, ticks, T* and the Eq. 1 barrier of the measured times."""
    import dataclasses

    import torch

    from . import aggregate
    from .rounds import OscarsRun
    K = cfg.K
    if schedule.K != K:
        raise ValueError("schedule and workload disagree on K")
    run = OscarsRun(dataclasses.replace(cfg, batch=schedule.max_batch), dataset, init)
    balancer = LoadBalancer(K, cfg.M, resolution)
    kinds = list(range(7))
    records = []
    tau = [1] * K
    try:
        for r in range(rounds):
            batches = schedule.at(r)
            ms = [0.0] * K
            for k in range(K):
                if tau[k] == 0:
                    continue
                solo = [0] * K
                solo[k] = tau[k]
                run.ctx.profile_begin(kinds)
                run.ctx.local_steps(run.replicas, run.x, run.y, run.offsets, run.seed, solo,
                                    cfg.lr, batches[k])
                prof = run.ctx.profile_end()
                ms[k] = float(sum(v[0] for v in prof.values()))
            aggregate(run.g, run.replicas, run.weights, K, run.n, run.n, True)
            t_iter = [m / a for m, a in zip(ms, tau)]
            rec = {"round": r, "tau": list(tau), "batches": batches, "gpu_ms": ms,
                   "t_iter_ms": t_iter, "barrier_ms": barrier_time(tau, t_iter),
                   "idle": idle_fraction(tau, t_iter)}
            balancer.update(t_iter)
            rec["next_ticks"], rec["next_T_star"] = list(balancer.ticks), balancer.T_star
            rec["next_tau"] = list(balancer.tau)
            records.append(rec)
            tau = list(balancer.tau)
        torch.cuda.synchronize()
        model = run.global_layers() if return_model else None
        cursors = run.ctx.cursors()
    finally:
        run.close()
    return {"records": records, "model": model, "cursors": cursors,
            "tau_changes": balancer.changes}


def time_to_loss(result: Dict, target: float) -> Optional[float]:
    """Emulated clock at the first evaluation at or below ``target``."""
    for rec in result["records"]:
        if "eval_loss" in rec and rec["eval_loss"] <= target:
            return rec["clock"]
    return None


def compare(cfg, schedule: SpeedSchedule, time_budget_steps: float, local_steps: int = 4,
            resolution: int = 8, n_eval: int = 10000, base: Optional[float] = None,
            eval_every: int = 1) -> Dict:
    """The three paradigms on one workload and one emulated cluster.  The
    budget is in units of the speed-1 step time."""
    import workload
    dataset = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    eval_set = workload.gen_eval_set(cfg, n_eval)
    base_ms = measure_step_ms(cfg, dataset, init) if base is None else float(base)
    budget = time_budget_steps * base_ms
    out = {"workload": cfg.name, "K": cfg.K, "batch": cfg.batch, "lr": cfg.lr,
           "speeds": schedule.speeds, "changes": {str(k): v for k, v in schedule.changes.items()},
           "jitter": schedule.jitter, "step_ms_speed1": base_ms, "time_budget_ms": budget,
           "local_steps": local_steps, "resolution": resolution, "M": cfg.M, "paradigms": {}}
    results = {}
    for p in PARADIGMS:
        t0 = time.perf_counter()
        res = run_paradigm(cfg, dataset, init, eval_set, p, schedule, base_ms, budget,
                           local_steps=local_steps, resolution=resolution,
                           eval_every=eval_every)
        res["wall_s"] = time.perf_counter() - t0
        results[p] = res
    # target: the best loss BSP reached within the budget
    target = min(rec["eval_loss"] for rec in results["bsp"]["records"] if "eval_loss" in rec)
    for p, res in results.items():
        recs = res["records"]
        last = recs[-1]
        last_eval = [rec for rec in recs if "eval_loss" in rec][-1]
        idle = [rec["idle"] for rec in recs if "idle" in rec]
        out["paradigms"][p] = {
            "rounds": len(recs) - 1, "clock_ms": last["clock"], "samples": res["samples"],
            "samples_per_clock_s": res["samples"] / (last["clock"] / 1e3) if last["clock"] else None,
            "final_eval_loss": last_eval["eval_loss"], "final_eval_acc": last_eval["eval_acc"],
            "final_eval_clock_ms": last_eval["clock"],
            "mean_idle": float(np.mean(idle)) if idle else None,
            "clock_to_bsp_best_loss_ms": time_to_loss(res, target),
            "tau_changes": res["tau_changes"], "gpu_ms": res["gpu_ms"],
            "gpu_samples_per_s": res["samples"] / (res["gpu_ms"] / 1e3) if res["gpu_ms"] else None,
            "curve": [(round(rec["clock"], 4), rec.get("eval_loss"), rec.get("eval_acc"))
                      for rec in recs if "eval_loss" in rec],
        }
    out["bsp_best_loss"] = target
    return out


def _measured_cfg():
    """The workload of the measured-time run: an fp32 MLP wide enough that a
    worker's step time grows with its mini-batch size."""
    import workload
    return workload.Config("measured-1024-2048-2048-10-fp32", (1024, 2048, 2048, 10), workload.FP32,
                           K=4, n_rows=8000, batch=1024, tau_rule="given", lr=0.02, seed=24,
                           mean_scale=0.3)


MEASURED_BATCHES = (64, 128, 512, 1024)


def main(argv=None):
    import workload
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--budget", type=float, default=400.0,
                    help="emulated time budget, in speed-1 step times")
    ap.add_argument("--local-steps", type=int, default=4)
    ap.add_argument("--resolution", type=int, default=8)
    ap.add_argument("--jitter", type=float, default=0.02)
    ap.add_argument("--mean-scale", type=float, default=0.1)
    ap.add_argument("--eval-every", type=int, default=1)
    ap.add_argument("--out", default=None, help="also write the JSON here")
    ap.add_argument("--measured", type=int, default=0, metavar="ROUNDS",
                    help="instead: this many rounds with the plan from measured times on the "
                         "1024-2048-2048-10 fp32 MLP, 4 workers with batches 64, 128, 512, 1024 "
                         "reversed half way")
    args = ap.parse_args(argv)
    if args.measured > 0:
        cfg = _measured_cfg()
        sched = BatchSchedule(MEASURED_BATCHES,
                              {args.measured // 2: tuple(reversed(MEASURED_BATCHES))})
        res = run_measured(cfg, workload.gen_dataset(cfg), workload.gen_init(cfg), sched,
                           args.measured, resolution=args.resolution)
        res.pop("model")
        line = json.dumps(res)
        print(line)
        if args.out:
            with open(args.out, "w") as f:
                f.write(line + "\n")
        return 0
    cfg = workload.scaled(workload.C2, mean_scale=args.mean_scale)
    schedule = SpeedSchedule(cfg.speeds, changes={args.budget / 2: tuple(reversed(cfg.speeds))},
                             jitter=args.jitter, seed=cfg.seed)
    res = compare(cfg, schedule, args.budget, local_steps=args.local_steps,
                  resolution=args.resolution, eval_every=args.eval_every)
    line = json.dumps(res)
    print(line)
    if args.out:
        with open(args.out, "w") as f:
            f.write(line + "\n")
    return 0


if __name__ == "__main__":
    sys.exit(main())
