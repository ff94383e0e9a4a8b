"""Benchmark of the Oscars local-SGD hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload c5]

A step is one Oscars round over the whole hot path: Algorithm 1 (tau from the
workers' iteration times), the mini-batch index table, tau_k local SGD steps
of every simulated worker (forward, loss gradient, backward-data,
backward-weight + SGD update, finished workers masked out), and the
parameter-server aggregation into the global model, all in one
oscars_round (every worker's first step reads the global model, so no
broadcast copies are written).  Inputs are resident in HBM before the timed
region.  Prints one JSON line.

Default workload: MLP 4096-4096-4096-4096-1000, bf16 inputs/weights with fp32
accumulation and fp32 masters, K = 8 workers with speed factors
1,1,2,2,3,4,6,8, batch 256, 200k-sample 1000-class Gaussian mixture, plus the
aggregation of the 54.4M-parameter model every round.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3}
PMC_FILE = os.path.join(ROOT, "profiles", "pmc_traffic.json")


def gemm_work(cfg, tau, fused_path=None):
    """Algorithmic FLOPs and bytes of every launch of one round (oscars_round),
    per kind.  Bytes: each operand read once, each result written once (weights
    bf16 in the products of bf16 workloads; fp32 master read and write in the
    update, and the bf16 copy for workers that take another step; the start
    model cast to bf16 once; the average reads K replicas and writes the
    global model).  A hidden layer whose backward is fused (backward-data +
    backward-weight + update in one launch; fused_path(l, ns), else every
    hidden layer of a bf16 model with batches up to 256) counts both products
    and the update's bytes plus the delta written for the layer below."""
    import numpy as np
    es = 2 if cfg.dtype == "bf16" else 4
    B, dims = cfg.batch, cfg.dims
    L = len(dims) - 1
    if fused_path is None:
        fused_path = lambda l, ns: cfg.dtype == "bf16" and B <= 256
    work = {"gemm_fwd": [0.0, 0.0], "gemm_dgrad": [0.0, 0.0], "gemm_wgrad_update": [0.0, 0.0],
            "gemm_bwd_fused": [0.0, 0.0], "softmax_ce": [0.0, 0.0], "cast_bf16": [0.0, 0.0],
            "aggregate": [0.0, 0.0]}
    tau = np.asarray(tau)
    n_params = sum(o * i + o for i, o in zip(dims[:-1], dims[1:]))
    if cfg.dtype == "bf16":
        work["cast_bf16"][1] += n_params * 6.0
    work["aggregate"][1] += (cfg.K + 1) * n_params * 4.0
    for j in range(int(tau.max())):
        ns = int((tau > j).sum())
        ns_next = int((tau > j + 1).sum())  # workers whose bf16 copy is refreshed
        for l in range(1, L + 1):
            i, o = dims[l - 1], dims[l]
            out_es = es if l < L else 4
            work["gemm_fwd"][0] += ns * 2.0 * B * o * i
            work["gemm_fwd"][1] += ns * (es * o * i + 4 * o + es * B * i + out_es * B * o)
            update = (ns * (8.0 * (o * i + o) + es * B * o + es * B * i)
                      + (ns_next * 2.0 * o * i if es == 2 else 0.0))
            if l > 1 and fused_path(l, ns):
                work["gemm_bwd_fused"][0] += ns * 4.0 * B * o * i
                work["gemm_bwd_fused"][1] += update + ns * es * B * i
                continue
            if l > 1:
                work["gemm_dgrad"][0] += ns * 2.0 * B * o * i
                work["gemm_dgrad"][1] += ns * (es * o * i + es * B * o + 2 * es * B * i)
            work["gemm_wgrad_update"][0] += ns * 2.0 * B * o * i
            work["gemm_wgrad_update"][1] += update
        C = dims[-1]
        work["softmax_ce"][1] += ns * B * (4 * C + es * C)
    return work


def head_fused(hw, c, classes):
    """Whether the library runs the classifier head of a local step as one
    launch: the last conv activation of a batch row, its pooled vector, its
    pooling gradient and the logits fit one workgroup's LDS (12288 floats)."""
    return hw * c + 2 * c + classes <= 12288


def cnn_work(cfg, tau, fused_path=None):
    """Algorithmic FLOPs and bytes of one round of the convolutional workload
    (oscars_round), per kind: conv layers as implicit GEMMs (2 FLOPs per
    multiply-add of every kernel tap; bytes: input, weights and output once),
    the classifier head (pooling, classifier, softmax and their backward-data)
    as softmax_ce where it is one launch, else pooling and the classifier with
    the forward and backward-data kinds; the weight updates' fp32 read and
    write of their parameters."""
    import numpy as np
    B = cfg.batch
    tau = np.asarray(tau)
    work = {k: [0.0, 0.0] for k in ("gemm_fwd", "gemm_dgrad", "gemm_wgrad_update", "softmax_ce",
                                    "aggregate", "gemm_bwd_fused")}
    H, W, C = cfg.image
    geo = []
    skips = list(cfg.skips or [False] * len(cfg.conv)) + [False]
    for co, st, *_ in cfg.conv:
        Ho, Wo = (H - 1) // st + 1, (W - 1) // st + 1
        geo.append((H, W, C, Ho, Wo, co))
        H, W, C = Ho, Wo, co
    classes = cfg.n_classes
    work["aggregate"][1] += (cfg.K + 1) * cfg.n_params * 4.0
    for j in range(int(tau.max())):
        ns = int((tau > j).sum())
        for l, (h, w, c, ho, wo, co) in enumerate(geo):
            macs = B * ho * wo * co * 9 * c
            act_in, act_out, wts = B * h * w * c * 4, B * ho * wo * co * 4, (9 * c * co + co) * 4
            work["gemm_fwd"][0] += ns * 2.0 * macs
            # a shortcut layer also reads its block's input (the shape of its output)
            work["gemm_fwd"][1] += ns * (act_in + wts + act_out * (2 if skips[l] else 1))
            # backward-data and backward-weight of conv layer l + 1 in one launch
            # (fused_path, the library's choice: one or two replicas), booked as
            # gemm_bwd_fused; the update stays with gemm_wgrad_update
            pair = l > 0 and fused_path is not None and fused_path(l + 1, ns)
            dk = "gemm_bwd_fused" if pair else "gemm_dgrad"
            wk = "gemm_bwd_fused" if pair else "gemm_wgrad_update"
            if l > 0:
                work[dk][0] += ns * 2.0 * macs
                # reads the mask too, and, below a shortcut, the shortcut's gradient
                work[dk][1] += ns * (act_out + wts + (3 if skips[l + 1] else 2) * act_in)
            work[wk][0] += ns * 2.0 * macs
            work[wk][1] += ns * (act_out + act_in)
            work["gemm_wgrad_update"][1] += ns * 2 * wts
        pooled, act, fc = B * C * 4, B * H * W * C * 4, (C * classes + classes) * 4
        if head_fused(H * W, C, classes):
            # one launch (booked as softmax_ce): the last activation read once, pooled,
            # logits, loss, delta and the gradient at the last conv output written
            work["softmax_ce"][0] += ns * 4.0 * B * C * classes
            work["softmax_ce"][1] += ns * (2 * act + pooled + fc + 2 * B * classes * 4)
        else:
            work["gemm_fwd"][1] += ns * (act + pooled)  # pooling
            work["gemm_fwd"][0] += ns * 2.0 * B * C * classes
            work["gemm_fwd"][1] += ns * (pooled + fc + B * classes * 4)
            work["gemm_dgrad"][0] += ns * 2.0 * B * C * classes
            work["gemm_dgrad"][1] += ns * (B * classes * 4 + C * classes * 4 + pooled)
            work["gemm_dgrad"][1] += ns * (pooled + 2 * act)  # pooling backward
            work["softmax_ce"][1] += ns * B * classes * 8
        work["gemm_wgrad_update"][0] += ns * 2.0 * B * C * classes
        work["gemm_wgrad_update"][1] += ns * (B * classes * 4 + pooled + 2 * fc)
    return work


def kernel_source_hash() -> str:
    p = os.path.join(ROOT, "paper_2102_08550_amd", "csrc", "kernels.hip")
    return hashlib.sha256(open(p, "rb").read()).hexdigest()[:16]


MIX_TOLERANCE = 0.05


def pmc_traffic(kernel: str, workload_name: str, algorithmic_bytes: float, mix=None,
                mix_bytes=None):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary, if it was taken on the current kernel source and on a launch mix
    close to this run's; else None.  The summary holds measured / algorithmic
    bytes per launch (FETCH_SIZE over the fetch pass's algorithmic bytes plus
    WRITE_SIZE over the write pass's); the ratio times this run's algorithmic
    bytes per launch gives the bytes.  Where the summary records its backward
    path per layer and active replica count and it differs from this run's
    (`mix`), the kind's algorithmic bytes per round under the two mixes
    (`mix_bytes(mix)`) must agree within MIX_TOLERANCE."""
    try:
        data = json.load(open(PMC_FILE))
    except (OSError, ValueError):
        return None
    ent = data.get(workload_name, {}).get(kernel)
    if not ent or ent.get("kernels_sha256_16") != kernel_source_hash() or not ent.get("ratio"):
        return None
    theirs = ent.get("backward_mix")
    if mix is not None and theirs is not None and theirs != mix:
        if mix_bytes is None or "schedule" in theirs or "schedule" in mix:
            return None
        ours, other = mix_bytes(mix), mix_bytes(theirs)
        if not ours or abs(other - ours) > MIX_TOLERANCE * ours:
            return None
    return ent["ratio"] * algorithmic_bytes


def host_info():
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        aff = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        aff = None
    return {"cpu_model": model, "os_cpu_count": os.cpu_count(), "affinity": aff,
            "note": "numpy matmul uses its BLAS threads ('cores'); elementwise numpy is one thread"}


def cpu_baseline(cfg, ds, init, tau, budget_s: float):
    """The oracle as it stands, on the host cores: the workers' local SGD steps
    of round after round (worker by worker, each from the initial model of the
    round, as a worker runs them), until the time budget is used; and the
    oracle aggregation on a slice of K replicas."""
    import numpy as np

    import oracle
    import workload
    try:
        from threadpoolctl import threadpool_info
        threads = max(i.get("num_threads", 1) for i in threadpool_info()) or 1
    except Exception:
        threads = os.cpu_count() or 1
    off = oracle.shard_offsets(cfg.n_rows, cfg.K)
    seed = workload.sampler_seed(cfg)
    x0 = [(W.astype(np.float64), b.astype(np.float64)) for W, b in init]
    cache = {}
    steps, rounds = 0, 0
    done = [0] * cfg.K
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < budget_s:
        for k in sorted(range(cfg.K), key=lambda k: -int(tau[k])):
            x = x0
            for j in range(int(tau[k])):
                rows = oracle.batch_rows(seed, off, k, done[k] + j, cfg.batch, cache)
                xb = workload.bf16_bits_to_f32(ds.x[rows]) if cfg.dtype == "bf16" else ds.x[rows]
                if cfg.is_cnn:
                    x, _ = oracle.cnn.sgd_step(x, xb.astype(np.float64), ds.y[rows], cfg.lr,
                                               cfg.image, cfg.strides, cfg.skips)
                else:
                    x, _ = oracle.sgd_step(x, xb.astype(np.float64), ds.y[rows], cfg.lr,
                                           cfg.dtype == "bf16")
                steps += 1
                if time.perf_counter() - t0 > budget_s:
                    break
            done[k] += int(tau[k])
            if time.perf_counter() - t0 > budget_s:
                break
        rounds += 1
    dt = time.perf_counter() - t0
    n_slice = 4_000_000
    reps = [np.random.default_rng(i).standard_normal(n_slice).astype(np.float32)
            for i in range(cfg.K)]
    t1 = time.perf_counter()
    oracle.tree_aggregate(reps, oracle.paper_weights(cfg.K))
    dta = time.perf_counter() - t1
    return {
        "value": steps * cfg.batch / dt, "unit": "samples/s", "cores": threads, "kind": "oracle",
        "host": host_info(),
        "sample": f"{steps} local SGD steps of batch {cfg.batch} (workers' steps of {rounds} "
                  f"round(s), each worker from the round's start model; {dt:.1f} s, float64"
                  f"{' with bf16 rounding points' if cfg.dtype == 'bf16' else ''}); aggregation of "
                  f"{cfg.K} x {n_slice} fp32 slices",
        "aggregate_GBps": (cfg.K + 1) * n_slice * 4 / dta / 1e9,
    }


def bench_aggregation(args, cfg, copy):
    """Aggregation stress: K = 32 replicas of 25.6M fp32.  Before each round
    (untimed) the replicas are rebuilt as g + delta_k; the aggregate +
    broadcast launch of each round is timed with events on the same stream."""
    import numpy as np
    import torch

    import oracle
    import workload
    import paper_2102_08550_amd as P
    print(f"[bench] generating {cfg.name}", file=sys.stderr, flush=True)
    g0, delta = workload.gen_agg_vectors(cfg)
    stale = workload.gen_staleness(cfg)
    n, K = cfg.n_flat, cfg.K
    G = torch.from_numpy(g0).cuda()
    D = torch.from_numpy(delta).cuda()
    del delta
    R = torch.empty_like(D)
    stream = torch.cuda.current_stream()
    evs = []
    for s in range(args.warmup + args.steps):
        w = P.paper_weights(K, stale[s % cfg.rounds])
        torch.add(G.unsqueeze(0), D, out=R)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        P.aggregate(G, R, w, K, n, n, True)
        e1.record(stream)
        if s >= args.warmup:
            evs.append((e0, e1))
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(b) for a, b in evs)
    bytes_round = (2 * K + 1) * n * 4.0
    gbps = bytes_round * args.steps / (ms / 1e3) / 1e9
    out = {
        "metric": "local-SGD samples/sec (K sim workers, 1 GPU); aggregation GB/s vs HBM peak",
        "value": gbps, "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms / args.steps, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic (seeded N(0,1) + N(0,0.02^2))",
        "config": {"workload": cfg.name, "K": K, "n": n, "broadcast": True},
        "roofline": {"bound": "hbm", "achieved": gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": gbps / HBM_PEAK_GBPS,
                     "traffic": pmc_traffic("aggregate", args.workload, bytes_round),
                     "kernel": "aggregate",
                     "avg_launch_us": ms * 1000.0 / args.steps,
                     "algorithmic_per_launch": {"flop": 0.0, "bytes": bytes_round},
                     "achieved_vs_copy": gbps / copy["GBps"]},
        "hbm_copy": copy,
    }
    if args.cpu_budget > 0:
        m = 4_000_000
        xs = [np.random.default_rng(k).standard_normal(m).astype(np.float32) for k in range(K)]
        t0 = time.perf_counter()
        oracle.tree_aggregate(xs, oracle.paper_weights(K))
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": (K + 1) * m * 4 / dt / 1e9, "unit": "GB/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"oracle tree aggregation of {K} x {m} fp32 (no broadcast)"}
    print(json.dumps(out), flush=True)


def hbm_copy_probe(mib: int = 1024, reps: int = 5):
    """Practical HBM ceiling of a plain fp32 copy of ``mib`` MiB (read + write
    bytes over the mean time of ``reps`` copies after one warm copy), with
    torch's device-to-device copy and with the library's broadcast at K = 1
    (non-temporal stores); the faster one is the ceiling."""
    import torch

    import paper_2102_08550_amd as P
    n = mib * (1 << 20) // 4
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return 2 * n * 4 / (a.elapsed_time(b) / reps / 1e3) / 1e9

    torch_gbps = timed(lambda: dst.copy_(src))
    nt_gbps = timed(lambda: P.broadcast(src, dst, 1, n, n))
    assert torch.equal(dst, src)
    del src, dst
    gbps = max(torch_gbps, nt_gbps)
    return {"GBps": gbps, "frac_spec_peak": gbps / HBM_PEAK_GBPS, "bytes": 2 * n * 4,
            "torch_copy_GBps": torch_gbps, "broadcast_K1_GBps": nt_gbps,
            "what": f"fp32 copy of {mib} MiB (read + write), mean of {reps}: torch's "
                    "device-to-device copy and oscars_broadcast with K = 1; the faster"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c5",
                    choices=["c1", "c2", "c3", "c4", "c5", "c6", "c7"],
                    help="c5 (default): the full round; c4: aggregation-only stress; c6: the "
                         "convolutional workload; c7: its ResNet-style variant (residual blocks)")
    ap.add_argument("--cpu-budget", type=float, default=20.0,
                    help="seconds of oracle work for the CPU baseline (0 = skip)")
    ap.add_argument("--backward", default="auto", choices=["auto", "separate", "fused",
                                                           "fused_split"],
                    help="backward path of the hidden bf16 layers (auto: timed per "
                         "configuration in this process; a fixed one makes counter passes of "
                         "separate processes run the same launch mix)")
    ap.add_argument("--schedule", default="grouped", choices=["grouped", "replica"],
                    help="grouped (default): one oscars_round, every local step of all active "
                         "workers in one launch per layer and pass; replica: the same round "
                         "worker after worker (a broadcast, each worker's tau_k steps alone, "
                         "then the average), to measure a replica-major order")
    ap.add_argument("--probe-copy-mib", type=int, default=0,
                    help="first run a plain device-to-device copy of this many MiB, three "
                         "times (calibration of hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "the hot path runs on one GPU; --gpus must be 1"}))
        sys.exit(2)

    import numpy as np
    import torch

    import workload
    import paper_2102_08550_amd as P
    from paper_2102_08550_amd.rounds import OscarsRun

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.probe_copy_mib > 0:
        n = args.probe_copy_mib * (1 << 20) // 4
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    copy = hbm_copy_probe()
    cfg = workload.CONFIGS[args.workload]
    if args.workload == "c4":
        return bench_aggregation(args, cfg, copy)
    print(f"[bench] generating {cfg.name}", file=sys.stderr, flush=True)
    ds = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    stream = torch.cuda.current_stream()
    run = OscarsRun(cfg, ds, init, stream=stream)
    run.ctx.set_backward(P.BACKWARDS[args.backward])

    def do_round(tau):
        if args.schedule == "grouped":
            run.round(tau)
            return
        # replica-major: every worker's steps back to back, from the global model
        P.broadcast(run.g, run.replicas, cfg.K, run.n, run.n)
        for k in sorted(range(cfg.K), key=lambda k: -int(tau[k])):
            solo = [0] * cfg.K
            solo[k] = int(tau[k])
            run.local_steps(solo)
        P.aggregate(run.g, run.replicas, run.weights, cfg.K, run.n, run.n, False)

    def tau_for(step):
        if cfg.tau_rule == "speeds":  # Algorithm 1 from the workers' iteration times
            return P.load_balance(workload.speeds_to_t_iter(cfg.speeds), cfg.M)[1]
        if cfg.tau_rule == "given":
            return list(cfg.tau_given)
        draws = workload.gen_tau_uniform(cfg)
        return draws[step % len(draws)].tolist()

    kinds = [P.KERNEL_CAST, P.KERNEL_FWD, P.KERNEL_SOFTMAX, P.KERNEL_DGRAD, P.KERNEL_WGRAD,
             P.KERNEL_AGGREGATE, P.KERNEL_BWD_FUSED]
    # Warmup rounds carry HIP events around every launch: the per-kernel
    # breakdown, and which kernel dominates.  The timed rounds carry events
    # around the dominant kernel's launches only (events around every launch
    # would add about 10% to a round).
    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    # The first rounds pick the forward / backward-data GEMM tilings (the
    # launches of each configuration run the candidate tilings in turn until
    # the fastest is kept) and the backward path (timed at its first launch);
    # they are neither profiled nor timed.
    n_tune = 0
    while True:
        do_round(tau_for(n_tune))
        n_tune += 1
        if run.ctx.tuning_pending() == 0 or n_tune >= 64:
            break
    torch.cuda.synchronize()
    print(f"[bench] {n_tune} tuning rounds", file=sys.stderr, flush=True)

    def fused_path(l, ns):  # the backward path the library took (timed in the first round)
        return run.ctx.backward_path(l, cfg.batch, ns) == 1

    run.ctx.profile_begin(kinds)
    work_w = {}
    n_warm = max(args.warmup, 2) - 1
    samples_w = 0
    for s in range(1, n_warm + 1):
        tau = tau_for(s)
        do_round(tau)
        samples_w += int(np.sum(tau)) * cfg.batch
        for kname, (fl, by) in (cnn_work(cfg, tau, fused_path) if cfg.is_cnn
                                else gemm_work(cfg, tau, fused_path)).items():
            a = work_w.setdefault(kname, [0.0, 0.0])
            a[0] += fl
            a[1] += by
    prof_w = run.ctx.profile_end()
    dom = max((k for k in prof_w if prof_w[k][1] > 0), key=lambda k: prof_w[k][0])
    dom_kind = P.KERNEL_NAMES.index(dom)

    samples = 0
    work_tot = {}
    # The last timed round carries HIP events around the dominant kernel's
    # launches (every round runs the same launch sequence).
    print(f"[bench] timing {args.steps} rounds (events around {dom} in the last)", file=sys.stderr,
          flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        tau = tau_for(args.warmup + s)
        if s == args.steps - 1:
            run.ctx.profile_begin([dom_kind])
        do_round(tau)
        if s == args.steps - 1:
            work_tot = cnn_work(cfg, tau, fused_path) if cfg.is_cnn else gemm_work(cfg, tau, fused_path)
        samples += int(np.sum(tau)) * cfg.batch
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof = run.ctx.profile_end()
    elapsed = t1 - t0
    ms_per_step = elapsed * 1000.0 / args.steps

    def summarize(prof_, work_, rounds):
        out_ = {}
        for name, (ms, cnt) in prof_.items():
            if cnt == 0:
                continue
            fl, by = work_.get(name, [0.0, 0.0])
            out_[name] = {"ms": ms, "ms_per_round": ms / rounds, "launches": cnt,
                          "avg_us": ms * 1000.0 / cnt,
                          "TFLOPs": fl / (ms / 1e3) / 1e12 if fl else None,
                          "GBps": by / (ms / 1e3) / 1e9 if by else None,
                          "flop_per_launch": fl / cnt, "bytes_per_launch": by / cnt}
        return out_
    kernels = summarize(prof_w, work_w, n_warm)  # breakdown (warmup, every kernel timed)
    d = summarize(prof, work_tot, 1)[dom]  # dominant kernel, inside the timed region
    ridge = MFMA_PEAK_TFLOPS[cfg.dtype] * 1e12 / (HBM_PEAK_GBPS * 1e9)
    intensity = d["flop_per_launch"] / d["bytes_per_launch"] if d["bytes_per_launch"] else 0.0
    if intensity > ridge:
        roof = {"bound": "mfma", "achieved": d["TFLOPs"], "peak": MFMA_PEAK_TFLOPS[cfg.dtype],
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": d["GBps"], "peak": HBM_PEAK_GBPS, "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    tau0 = np.asarray(tau_for(0))
    backward_mix = {f"l{l}": {str(ns): ("fused" if fused_path(l, ns) else "separate")
                              for ns in sorted({int((tau0 > j).sum()) for j in range(tau0.max())})}
                    for l in range(1, (len(cfg.conv) + 2) if cfg.is_cnn else len(cfg.dims))}
    mix = backward_mix if args.schedule == "grouped" else {"schedule": "replica"}

    def mix_bytes(m):  # the dominant kind's algorithmic bytes per round under mix m
        if cfg.is_cnn:
            return cnn_work(cfg, tau0, fused_path)[dom][1]
        path = lambda l, ns: m.get(f"l{l}", {}).get(str(ns), "fused") == "fused"  # noqa: E731
        return gemm_work(cfg, tau0, path)[dom][1]
    roof["traffic"] = pmc_traffic(dom, args.workload, d["bytes_per_launch"], mix, mix_bytes)
    if roof["traffic"] is not None:
        roof["traffic_basis"] = ("committed counter passes' measured/algorithmic bytes per launch "
                                 "x this run's algorithmic bytes per launch")
    roof["kernel"] = dom
    roof["avg_launch_us"] = d["avg_us"]
    roof["algorithmic_per_launch"] = {"flop": d["flop_per_launch"], "bytes": d["bytes_per_launch"]}

    local_ms = sum(v["ms"] for k, v in kernels.items() if k != "aggregate")
    flops = sum(v[0] for k, v in work_w.items() if k != "aggregate")
    out = {
        "metric": "local-SGD samples/sec (K sim workers, 1 GPU); aggregation GB/s vs HBM peak",
        "value": samples / elapsed,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded Gaussian mixture, random init)",
        "config": {"workload": cfg.name, "dims": list(cfg.dims), "K": cfg.K, "batch": cfg.batch,
                   "tau": tau_for(0), "lr": cfg.lr, "n_params": cfg.n_params,
                   "samples_per_round": samples // args.steps, "parallelism": "1 GPU, K simulated"},
        "kernels_note": "per-kernel breakdown from the warmup rounds (events around every "
                        "launch); the roofline kernel is timed by events around its launches "
                        "in the last timed round",
        "aggregation": ({"GBps": kernels["aggregate"]["GBps"],
                         "frac_hbm_peak": kernels["aggregate"]["GBps"] / HBM_PEAK_GBPS,
                         "avg_us": kernels["aggregate"]["avg_us"],
                         "bytes_per_round": kernels["aggregate"]["bytes_per_launch"],
                         "note": "K-way average into the global model; oscars_round starts the "
                                 "next round's workers from it, so no broadcast copies are "
                                 "written"}
                        if "aggregate" in kernels else None),
        "local_steps": {"kernel_ms_per_round": local_ms / n_warm,
                        "TFLOPs": flops / (local_ms / 1e3) / 1e12 if local_ms else None,
                        "frac_mfma_peak": flops / (local_ms / 1e3) / 1e12 / MFMA_PEAK_TFLOPS[cfg.dtype]
                        if local_ms else None,
                        "samples_per_s_kernels": samples_w / (local_ms / 1e3) if local_ms else None},
        "kernels": kernels,
        "backward": {"mode": args.backward, "path_per_layer_and_active_replicas": backward_mix},
        "schedule": args.schedule,
        "roofline": roof,
        "hbm_copy": copy,
    }
    roof["achieved_vs_copy"] = roof["achieved"] / copy["GBps"] if roof["unit"] == "GB/s" else None
    losses = run.ctx.round_losses()
    out["last_round_mean_loss"] = float(np.nanmean(losses))
    run.close()
    if args.cpu_budget > 0:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(cfg, ds, init, np.asarray(tau_for(0)), args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
