"""GPU parity of the local SGD steps (Approach, Eq. 4, second branch) and of
whole rounds against the oracle, on the same seeded inputs.

Trajectories are compared tensor by tensor (each W_l and b_l), element by
element: the norm-wise relative error of the difference and its largest
element relative to the tensor's largest element, both within the tolerance.
The small workloads run at full size, the large ones with their layer widths
scaled down (tiles still ragged in M, N and K), and batches above 256 and
more than 1024 classes have cases of their own.  The full-size C3 and C5
workloads run all their rounds in the launch configuration the benchmark
times and are compared with the oracle's run of the same rounds, stored in
tests/golden/full_size_*.npz by tests/golden/make_full_size.py.  The achieved
agreement of every case is written to gpurun_out/parity/."""
import numpy as np
import pytest

import oracle
import workload
from _parity import (BF16_TOL, FP32_TOL, assert_tensors_close, gpu_rounds, oracle_rounds,
                     oracle_tau, record, rel_err, say, tensor_errors)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2102_08550_amd
    return paper_2102_08550_amd


TRAJ = {
    "c1": workload.C1,
    "c2": workload.C2,
    "c3s": workload.scaled(workload.C3, dims=(3072, 264, 136, 10), n_rows=6400, rounds=4),
    "c5s": workload.scaled(workload.C5, dims=(512, 392, 264, 200, 1000), n_rows=16000, rounds=3,
                           batch=72),
    "tiny-fp32": workload.Config("tiny-fp32", (8, 3), workload.FP32, K=3, n_rows=7, batch=1,
                                 tau_rule="given", tau_given=(0, 2, 5), lr=0.3, rounds=3, seed=9),
    "tiny-bf16": workload.Config("tiny-bf16", (16, 24, 37), workload.BF16, K=3, n_rows=40,
                                 batch=5, tau_rule="given", tau_given=(4, 0, 1), lr=0.2, rounds=3,
                                 seed=10),
    "k1-sgd": workload.Config("k1-sgd", (40, 136, 10), workload.FP32, K=1, n_rows=300, batch=33,
                              tau_rule="given", tau_given=(1,), lr=0.1, rounds=12, seed=11),
    # Batches above 128 take the whole-batch tiles; K of 2056 and 1040 is
    # three and two K chunks (the last one ragged), split over workgroups at
    # these replica counts.
    "wide-bf16": workload.Config("wide-bf16", (2056, 1032, 264, 100), workload.BF16, K=4,
                                 n_rows=3000, batch=256, tau_rule="given", tau_given=(3, 1, 2, 4),
                                 lr=0.05, rounds=2, seed=13),
    "wide-fp32": workload.Config("wide-fp32", (1040, 2056, 136, 10), workload.FP32, K=3,
                                 n_rows=1500, batch=160, tau_rule="given", tau_given=(2, 3, 1),
                                 lr=0.05, rounds=2, seed=14),
    # Batch above 256 (bf16: the separate backward, two whole-batch N tiles,
    # the second ragged) and more than 1024 classes (the softmax walks the
    # row in column blocks).
    "b300-c1100-bf16": workload.Config("b300-c1100-bf16", (264, 520, 1100), workload.BF16, K=3,
                                       n_rows=2400, batch=300, tau_rule="given",
                                       tau_given=(2, 1, 3), lr=0.05, rounds=2, seed=21),
    # The largest batch the library accepts, fp32, 1030 classes.
    "b1024-c1030-fp32": workload.Config("b1024-c1030-fp32", (72, 136, 1030), workload.FP32, K=2,
                                        n_rows=4100, batch=1024, tau_rule="given",
                                        tau_given=(1, 2), lr=0.05, rounds=2, seed=22),
}


TRAJ_CASES = [(n, False) for n in TRAJ] + [("c2", True), ("c5s", True), ("tiny-bf16", True)]


@pytest.mark.parametrize("name,fused", TRAJ_CASES,
                         ids=[f"{n}-{'round' if f else 'steps+agg'}" for n, f in TRAJ_CASES])
def test_trajectory_matches_oracle(P, name, fused):
    cfg = TRAJ[name]
    say(f"trajectory {name} fused={fused}: dims={cfg.dims} K={cfg.K} B={cfg.batch} R={cfg.rounds}")
    ds = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    from paper_2102_08550_amd.rounds import tau_schedule
    tau = tau_schedule(cfg)
    assert np.array_equal(tau, oracle_tau(cfg, cfg.rounds))
    g_gpu, l_gpu = gpu_rounds(cfg, ds, init, tau, fused=fused)
    g_ref, l_ref = oracle_rounds(cfg, ds, init, tau)
    tol = BF16_TOL if cfg.dtype == workload.BF16 else FP32_TOL
    per_round = [tensor_errors(a, b) for a, b in zip(g_gpu, g_ref)]
    loss_err = [[abs(float(l_gpu[r][k]) - l_ref[r][k]) / max(abs(l_ref[r][k]), 1e-2)
                 if tau[r][k] > 0 else None for k in range(cfg.K)] for r in range(cfg.rounds)]
    worst = [max(max(e["rel"], e["max"]) for e in pr.values()) for pr in per_round]
    say(f"  worst per-tensor error per round: {[f'{e:.2e}' for e in worst]}")
    record(f"trajectory-{name}-{'round' if fused else 'steps'}",
           {"tol": tol, "tensors": per_round, "loss_rel": loss_err,
            "global_rel": [rel_err(a, b) for a, b in zip(g_gpu, g_ref)]})
    checkpoints = sorted({min(cfg.rounds, 10) - 1, cfg.rounds - 1})
    for r in checkpoints:
        assert_tensors_close(per_round[r], tol, f"round {r + 1}")
    for r in range(cfg.rounds):
        for k in range(cfg.K):
            if tau[r][k] == 0:
                assert np.isnan(l_gpu[r][k])
            else:
                assert loss_err[r][k] <= tol, (r, k, l_gpu[r][k], l_ref[r][k])


def _run_once(P, cfg, ds, init, tau_rounds, tiling=None, backward=None):
    import torch
    from paper_2102_08550_amd.rounds import OscarsRun
    run = OscarsRun(cfg, ds, init)
    if tiling is not None:
        run.ctx.set_gemm_tiling(tiling)
    if backward is not None:
        run.ctx.set_backward(backward)
    for tau in tau_rounds:
        run.local_steps([int(t) for t in tau])
    torch.cuda.synchronize()
    reps = run.replicas.view(cfg.K, run.n).cpu().numpy().copy()
    cur = run.ctx.cursors()
    run.close()
    return reps, cur


MASK_CFGS = [
    workload.scaled(workload.C5, dims=(256, 136, 200), n_rows=2000, rounds=1, batch=40, K=5,
                    tau_rule="given", tau_given=(3, 1, 0, 4, 2)),
    workload.scaled(workload.C2, dims=(64, 72, 10), n_rows=900, rounds=1, batch=17, K=4,
                    tau_rule="given", tau_given=(2, 5, 1, 3)),
    # 4096-wide layers at batch 256: 8, 4, 2 and 1 active replicas take the
    # 128 x 256 tile, the 64 x 256 tile, and split-K over either, while every
    # solo run takes the 1-replica launches; all must agree bit for bit.
    workload.scaled(workload.C5, dims=(4096, 4096, 1000), n_rows=4000, rounds=1, batch=256, K=8,
                    tau_rule="given", tau_given=(2, 1, 3, 1, 2, 1, 1, 4)),
]


@pytest.mark.parametrize("cfg", MASK_CFGS, ids=["bf16", "fp32", "bf16-wide"])
def test_masking_independence_and_determinism(P, cfg):
    """A replica's result does not depend on which other replicas run beside
    it (grouped == solo, bit for bit); tau_k = 0 leaves a replica untouched;
    two identical runs agree bit for bit."""
    say(f"masking {cfg.dtype} tau={cfg.tau_given}")
    ds = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    tau = np.array([cfg.tau_given])
    grouped, cur = _run_once(P, cfg, ds, init, tau)
    again, _ = _run_once(P, cfg, ds, init, tau)
    assert np.array_equal(grouped.view(np.uint32), again.view(np.uint32))
    assert cur == list(cfg.tau_given)
    from paper_2102_08550_amd import Context
    for k in range(cfg.K):
        solo_tau = np.zeros((1, cfg.K), np.int32)
        solo_tau[0, k] = cfg.tau_given[k]
        solo, _ = _run_once(P, cfg, ds, init, solo_tau)
        assert np.array_equal(solo[k].view(np.uint32), grouped[k].view(np.uint32)), k
    # tau = 0 replica equals the initial model
    ctx = Context(cfg.dims, 1 if cfg.dtype == "bf16" else 0, cfg.K, cfg.batch)
    flat = ctx.pack(init)
    ctx.close()
    for k in range(cfg.K):
        if cfg.tau_given[k] == 0:
            assert np.array_equal(grouped[k], flat)


TILING_CFGS = [
    MASK_CFGS[2],
    workload.Config("tiling-fp32", (1040, 2056, 136, 10), workload.FP32, K=3, n_rows=1500,
                    batch=160, tau_rule="given", tau_given=(2, 3, 1), lr=0.05, rounds=1,
                    seed=15),
]


@pytest.mark.parametrize("cfg", TILING_CFGS, ids=["bf16-wide", "fp32-wide"])
def test_every_tiling_gives_identical_results(P, cfg):
    """Every forward / backward-data tiling, split-K included, sums in the
    same order: the replicas after the local steps agree bit for bit with the
    automatically chosen tilings."""
    say(f"tilings {cfg.dtype} dims={cfg.dims} tau={cfg.tau_given}")
    ds = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    tau = np.array([cfg.tau_given])
    results = {}
    for name, t in P.TILINGS.items():
        results[name], _ = _run_once(P, cfg, ds, init, tau, tiling=t)
        say(f"  tiling {name} done")
    for name, reps in results.items():
        assert np.array_equal(reps.view(np.uint32), results["auto"].view(np.uint32)), name
    ctx = P.Context(cfg.dims, P.BF16 if cfg.dtype == "bf16" else P.FP32, 1, 8)
    for bad in (len(P.TILINGS), -1):
        with pytest.raises(P.OscarsError):
            ctx.set_gemm_tiling(bad)
    ctx.close()


def test_online_tiling_choice_settles(P):
    """AUTO tunes online: the launches of a configuration run the candidate
    tilings in turn until the fastest is kept, and the tuning ends; every
    launch gives the same bits, so the tuned run equals a run with one forced
    tiling round for round."""
    import torch
    from paper_2102_08550_amd.rounds import OscarsRun
    cfg = MASK_CFGS[2]
    say(f"online tiling {cfg.dtype} dims={cfg.dims} tau={cfg.tau_given}")
    ds = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    tau = [int(t) for t in cfg.tau_given]
    run = OscarsRun(cfg, ds, init)
    assert run.ctx.tuning_pending() == 0
    n = 0
    while True:
        run.local_steps(tau)
        n += 1
        torch.cuda.synchronize()
        if n == 1:
            assert run.ctx.tuning_pending() > 0
        elif run.ctx.tuning_pending() == 0:
            break
        assert n < 40, "tuning did not settle"
    auto = run.replicas.view(cfg.K, run.n).cpu().numpy().copy()
    run.close()
    say(f"  settled after {n} rounds")
    forced, _ = _run_once(P, cfg, ds, init, np.array([tau] * n), tiling=P.TILING_L)
    assert np.array_equal(auto.view(np.uint32), forced.view(np.uint32))


def test_contexts_tune_independently(P):
    """Tiling and backward settings belong to a context: a forced tiling or
    backward mode in one context, or a restart of its tuning, leaves another
    context's tuning and its results as they were."""
    import torch
    from paper_2102_08550_amd.rounds import OscarsRun
    cfg = MASK_CFGS[2]
    say(f"independent contexts {cfg.dtype} dims={cfg.dims} tau={cfg.tau_given}")
    ds = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    tau = [int(t) for t in cfg.tau_given]
    a = OscarsRun(cfg, ds, init)
    b = OscarsRun(cfg, ds, init)
    b.ctx.set_gemm_tiling(P.TILING_S)
    b.ctx.set_backward(P.BACKWARD_SEPARATE)
    a.local_steps(tau)
    b.local_steps(tau)
    torch.cuda.synchronize()
    pending_a = a.ctx.tuning_pending()
    assert pending_a > 0 and b.ctx.tuning_pending() == 0
    b.ctx.set_gemm_tiling(P.TILING_AUTO)  # restarts b's tuning only
    assert a.ctx.tuning_pending() == pending_a
    # a still takes its own (AUTO) backward path; b the separate launches
    L = len(cfg.dims) - 1
    assert b.ctx.backward_path(L, cfg.batch, 1) == 0
    assert a.ctx.backward_path(L, cfg.batch, 1) in (0, 1)
    assert torch.equal(a.replicas, b.replicas)
    a.close()
    b.close()


BACKWARD_CFGS = [
    # output features of 2056 and 1032: three and two chunks of 1024 (the last
    # ragged), input strips ragged (1032 = 16 x 64 + 8, 200), 37 classes;
    # batch 256 (split partials available for up to 4 replicas)
    workload.Config("bwd-wide", (136, 1032, 2056, 200, 37), workload.BF16, K=4, n_rows=2000,
                    batch=256, tau_rule="given", tau_given=(3, 1, 2, 4), lr=0.05, rounds=1,
                    seed=16),
    # batch 40 (not a multiple of 32), one worker idle
    workload.Config("bwd-b40", (72, 1040, 1032, 10), workload.BF16, K=3, n_rows=600, batch=40,
                    tau_rule="given", tau_given=(2, 0, 3), lr=0.1, rounds=1, seed=17),
    # batch 128 (two dgrad waves idle) and batch 1
    workload.Config("bwd-b128", (256, 2056, 136, 10), workload.BF16, K=2, n_rows=700, batch=128,
                    tau_rule="given", tau_given=(2, 1), lr=0.05, rounds=1, seed=18),
    workload.Config("bwd-b1", (64, 264, 72, 5), workload.BF16, K=2, n_rows=50, batch=1,
                    tau_rule="given", tau_given=(1, 3), lr=0.2, rounds=1, seed=19),
    # a 4096 x 4096 hidden layer at 6 and 2 active replicas: the automatic
    # choice gives each workgroup two of the four chunks of output features
    workload.Config("bwd-4096", (256, 4096, 4096, 10), workload.BF16, K=6, n_rows=1600,
                    batch=256, tau_rule="given", tau_given=(2, 1, 1, 2, 1, 1), lr=0.05, rounds=1,
                    seed=20),
]


@pytest.mark.parametrize("cfg", BACKWARD_CFGS, ids=[c.name for c in BACKWARD_CFGS])
def test_backward_modes_identical(P, cfg):
    """The fused backward of hidden bf16 layers (backward-data, backward-weight
    and update in one launch; unsplit or split over chunks of output
    features), and layer 1's update streamed the same way without
    backward-data, give the replicas of the separate launches bit for bit,
    over local steps that start from the replicas and from a global model."""
    import torch
    from paper_2102_08550_amd.rounds import OscarsRun
    say(f"backward modes {cfg.name} dims={cfg.dims} B={cfg.batch} tau={cfg.tau_given}")
    ds = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    tau = [int(t) for t in cfg.tau_given]
    results = {}
    for name, mode in P.BACKWARDS.items():
        run = OscarsRun(cfg, ds, init)
        run.ctx.set_backward(mode)
        run.round(tau)           # first step from the global model
        run.local_steps(tau)     # then from the replicas
        torch.cuda.synchronize()
        results[name] = (run.replicas.cpu().numpy().copy(), run.g.cpu().numpy().copy())
        if name == "auto":
            for bad in (len(P.BACKWARDS), -1):
                with pytest.raises(P.OscarsError):
                    run.ctx.set_backward(bad)
        run.close()
        say(f"  backward {name} done")
    ref_r, ref_g = results["separate"]
    assert np.isfinite(ref_r).all()
    for name, (r, g) in results.items():
        assert np.array_equal(r.view(np.uint32), ref_r.view(np.uint32)), name
        assert np.array_equal(g.view(np.uint32), ref_g.view(np.uint32)), name


def test_backward_path_reports_the_launches(P):
    """oscars_backward_path: AUTO has decided every (layer, active replicas)
    that a round ran; forced modes report their path (layer 1: the streamed
    update without backward-data, or the separate update); bad arguments are
    refused."""
    import torch
    from paper_2102_08550_amd.rounds import OscarsRun
    cfg = BACKWARD_CFGS[0]
    say(f"backward path {cfg.name} tau={cfg.tau_given}")
    ds = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    tau = [int(t) for t in cfg.tau_given]
    L = len(cfg.dims) - 1
    actives = sorted({sum(t > j for t in tau) for j in range(max(tau))})
    for name, mode in P.BACKWARDS.items():
        run = OscarsRun(cfg, ds, init)
        run.ctx.set_backward(mode)
        if mode == P.BACKWARD_AUTO:
            assert run.ctx.backward_path(2, cfg.batch, actives[0]) == -1  # not timed yet
        run.round(tau)
        torch.cuda.synchronize()
        for ns in actives:
            for l in range(1, L + 1):
                got = run.ctx.backward_path(l, cfg.batch, ns)
                want = {P.BACKWARD_SEPARATE: 0, P.BACKWARD_FUSED: 1,
                        P.BACKWARD_FUSED_SPLIT: 1}.get(mode, got)
                assert got in (0, 1) and got == want, (name, l, ns, got)
        for bad in ((0, cfg.batch, 1), (L + 1, cfg.batch, 1), (2, 0, 1),
                    (2, cfg.batch + 1, 1), (2, cfg.batch, 0), (2, cfg.batch, cfg.K + 1)):
            with pytest.raises(P.OscarsError):
                run.ctx.backward_path(*bad)
        run.close()


@pytest.mark.parametrize("dtype", [workload.BF16, workload.FP32])
def test_round_equals_local_steps_plus_aggregate(P, dtype):
    """oscars_round == (copy global into every replica, oscars_local_steps,
    oscars_aggregate without broadcast), bit for bit, over three rounds with a
    worker idle (tau = 0) in one of them."""
    import torch
    from paper_2102_08550_amd.rounds import OscarsRun
    cfg = workload.Config("round-eq", (72, 136, 64, 37), dtype, K=5, n_rows=900, batch=24,
                          tau_rule="given", lr=0.1, rounds=3, seed=12)
    ds = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    taus = [[3, 1, 0, 2, 4], [1, 1, 1, 1, 1], [2, 5, 3, 0, 1]]
    a = OscarsRun(cfg, ds, init)
    b = OscarsRun(cfg, ds, init)
    for t in taus:
        a.round(t)
        b.replicas.copy_(b.g.repeat(cfg.K))
        b.local_steps(t)
        b.aggregate(False)
        torch.cuda.synchronize()
        assert torch.equal(a.replicas, b.replicas)
        assert torch.equal(a.g, b.g)
        assert np.allclose(a.ctx.round_losses(), b.ctx.round_losses(), equal_nan=True)
    a.close()
    b.close()


def test_cursor_resume(P):
    """Two rounds in one context equal one round, then a fresh context given
    the saved cursors and replicas, then the second round (bit for bit)."""
    import torch
    from paper_2102_08550_amd.rounds import OscarsRun
    cfg = workload.scaled(workload.C3, dims=(128, 72, 10), n_rows=500, batch=24, K=4, rounds=2,
                          tau_rule="given")
    ds = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    taus = [[3, 1, 4, 2], [2, 5, 1, 3]]
    a = OscarsRun(cfg, ds, init)
    for t in taus:
        a.round(t)
    torch.cuda.synchronize()
    ref = a.g.cpu().numpy()
    cur_a = a.ctx.cursors()
    a.close()
    b = OscarsRun(cfg, ds, init)
    b.round(taus[0])
    saved_g = b.g.clone()
    saved_cur = b.ctx.cursors()
    b.close()
    c = OscarsRun(cfg, ds, init)
    c.g.copy_(saved_g)
    c.replicas.copy_(saved_g.repeat(cfg.K))
    c.ctx.set_cursors(saved_cur)
    c.round(taus[1])
    torch.cuda.synchronize()
    assert np.array_equal(c.g.cpu().numpy(), ref)
    assert c.ctx.cursors() == cur_a == [5, 6, 5, 5]
    c.close()


def test_local_steps_rejects_bad_arguments(P):
    import torch
    from paper_2102_08550_amd.rounds import OscarsRun
    cfg = workload.scaled(workload.C2, dims=(64, 72, 10), n_rows=400, batch=16, K=4, rounds=1,
                          tau_rule="given")
    ds = workload.gen_dataset(cfg)
    run = OscarsRun(cfg, ds, workload.gen_init(cfg))
    before = run.replicas.cpu().numpy().copy()
    ctx = run.ctx
    cases = [
        dict(tau=[1, -1, 1, 1]),
        dict(tau=[1, 1, 1, 5000]),
        dict(lr=0.0),
        dict(lr=float("nan")),
        dict(batch=17),  # above max_batch
        dict(batch=0),
        dict(offsets=[0, 100, 100, 300, 400]),  # empty shard
        dict(offsets=[0, 100, 200, 300, 399]),  # does not end at n_rows
    ]
    for c in cases:
        args = dict(tau=[1, 1, 1, 1], lr=0.1, batch=16, offsets=run.offsets)
        args.update(c)
        with pytest.raises(P.OscarsError) as ei:
            ctx.local_steps(run.replicas, run.x, run.y, args["offsets"], run.seed, args["tau"],
                            args["lr"], args["batch"])
        assert ei.value.status == P.E_INVALID, c
    torch.cuda.synchronize()
    assert np.array_equal(run.replicas.cpu().numpy(), before)
    assert ctx.cursors() == [0, 0, 0, 0]
    big = torch.zeros(cfg.K * run.n + 4, device="cuda")
    with pytest.raises(P.OscarsError):  # 4-byte aligned, not 16-byte aligned replicas
        ctx.local_steps(big[1:1 + cfg.K * run.n], run.x, run.y, run.offsets, run.seed, [1] * 4,
                        0.1, 16)
    run.close()
    with pytest.raises(P.OscarsError):  # width not a multiple of 8
        P.Context((60, 72, 10), P.FP32, 4, 16)
    with pytest.raises(P.OscarsError):
        P.Context((64, 72, 10), P.FP32, 65, 16)


def test_local_steps_refuse_graph_capture(P):
    """The local steps draw every call's batches on the host and wait for the
    previous call's index upload, so a stream being captured is refused with
    E_STATE before anything is enqueued; eager calls then go on unchanged."""
    import torch
    from paper_2102_08550_amd.rounds import OscarsRun
    cfg = workload.scaled(workload.C2, dims=(64, 72, 10), n_rows=400, batch=16, K=4, rounds=1,
                          tau_rule="given")
    ds = workload.gen_dataset(cfg)
    s = torch.cuda.Stream()
    run = OscarsRun(cfg, ds, workload.gen_init(cfg), stream=s)
    taus = [1, 2, 1, 3]
    run.round(taus)  # an earlier call whose upload the next one would wait for
    torch.cuda.synchronize()
    g_before, r_before = run.g.clone(), run.replicas.clone()
    cur = run.ctx.cursors()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s, capture_error_mode="relaxed"):
        with pytest.raises(P.OscarsError) as ei:
            run.round(taus)
        assert ei.value.status == P.E_STATE
        with pytest.raises(P.OscarsError) as ei:
            run.local_steps(taus)
        assert ei.value.status == P.E_STATE
    torch.cuda.synchronize()
    assert run.ctx.cursors() == cur
    assert torch.equal(run.g, g_before) and torch.equal(run.replicas, r_before)
    # the refused calls left no state behind: the next eager round matches a
    # fresh context resumed at the same cursors
    run.round(taus)
    ref = OscarsRun(cfg, ds, workload.gen_init(cfg))
    ref.g.copy_(g_before)
    ref.ctx.set_cursors(cur)
    ref.round(taus)
    torch.cuda.synchronize()
    assert torch.equal(run.g, ref.g)
    run.close()
    ref.close()


def _load_golden(name):
    import os
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                        f"full_size_{name}.npz")
    with np.load(path, allow_pickle=False) as z:
        return {k: z[k] for k in z.files}


@pytest.mark.parametrize("name", ["c3", "c5"])
def test_full_size_trajectory(P, name):
    """Full-size workload, all its rounds, in the benchmark's launch
    configuration (oscars_round), against the oracle's run of the same rounds:
      * every round, the average equals the oracle's tree over the GPU's own
        replicas bit for bit, each worker's mean loss agrees, and each
        tensor's norm and largest magnitude agree;
      * after rounds 1, R/2 and R, each tensor element by element on the
        stored indices (every element of the biases and of the small
        tensors, 8192 seeded positions of the others);
      * in round 1 the worker with the fewest steps is recomputed by the
        oracle in full and compared tensor by tensor, its update included."""
    import torch
    from paper_2102_08550_amd import Context
    from paper_2102_08550_amd.rounds import OscarsRun, tau_schedule
    cfg = workload.CONFIGS[name]
    gold = _load_golden(name)
    tol = BF16_TOL
    say(f"full-size {cfg.name}: generating data")
    ds = workload.gen_dataset(cfg)
    init = workload.gen_init(cfg)
    tau_all = tau_schedule(cfg)
    assert np.array_equal(tau_all, gold["tau"])
    checks = [int(c) for c in gold["check_rounds"]]
    run = OscarsRun(cfg, ds, init)
    unpack_ctx = Context(cfg.dims, P.BF16, 1, 1)
    log = {"tol": tol, "rounds": []}
    try:
        for r in range(cfg.rounds):
            tau = tau_all[r].tolist()
            say(f"  round {r + 1}/{cfg.rounds} tau={tau}")
            run.round(tau)
            losses = run.ctx.round_losses()
            torch.cuda.synchronize()
            reps = run.replicas.view(cfg.K, run.n).cpu().numpy()
            g = run.g.cpu().numpy()
            expect = oracle.tree_aggregate([reps[k] for k in range(cfg.K)],
                                           oracle.paper_weights(cfg.K))
            assert np.array_equal(g.view(np.uint32), expect.view(np.uint32)), \
                f"round {r + 1}: aggregate differs from the oracle tree"
            del expect
            entry = {"round": r + 1, "loss_rel": [], "norm_rel": {}, "absmax_rel": {}}
            for k in range(cfg.K):
                ref = float(gold["loss"][r][k])
                e = abs(float(losses[k]) - ref) / max(abs(ref), 1e-2)
                entry["loss_rel"].append(e)
                assert e <= tol, (r + 1, k, float(losses[k]), ref)
            layers = unpack_ctx.unpack(g)
            tensors = {}
            for l, (W, b) in enumerate(layers, start=1):
                tensors[f"W{l}"], tensors[f"b{l}"] = W.ravel(), b.ravel()
            for t, v in tensors.items():
                v64 = v.astype(np.float64)
                n_ref, m_ref = gold[f"norm_{t}"][r], gold[f"absmax_{t}"][r]
                entry["norm_rel"][t] = abs(np.linalg.norm(v64) - n_ref) / n_ref
                entry["absmax_rel"][t] = abs(np.abs(v64).max() - m_ref) / m_ref
                assert entry["norm_rel"][t] <= tol and entry["absmax_rel"][t] <= tol, \
                    (r + 1, t, entry["norm_rel"][t], entry["absmax_rel"][t])
            if r + 1 in checks:
                c = checks.index(r + 1)
                entry["sampled"] = {}
                for t, v in tensors.items():
                    ref = gold[f"val_{t}"][c].astype(np.float64)
                    got = v[gold[f"idx_{t}"]].astype(np.float64)
                    d = np.abs(got - ref)
                    e = {"rel": float(np.linalg.norm(d) / np.linalg.norm(ref)),
                         "max": float(d.max() / gold[f"absmax_{t}"][r]), "n": int(ref.size)}
                    entry["sampled"][t] = e
                assert_tensors_close(entry["sampled"], tol, f"round {r + 1}")
            if r == 0:
                k = int(np.argmin(tau))
                say(f"  oracle recomputes worker {k} ({tau[k]} steps) of round 1")
                off = oracle.shard_offsets(cfg.n_rows, cfg.K)
                x_ref, loss_ref = oracle.worker_local_steps(
                    [(W.astype(np.float64), b.astype(np.float64)) for W, b in init], ds.x_f32(),
                    ds.y, off, workload.sampler_seed(cfg), k, 0, int(tau[k]), cfg.lr, cfg.batch,
                    True)
                got = unpack_ctx.unpack(reps[k])
                errs = tensor_errors(got, x_ref)
                upd = tensor_errors([(a - W0, c - b0) for (a, c), (W0, b0) in zip(got, init)],
                                    [(a - W0, c - b0) for (a, c), (W0, b0) in zip(x_ref, init)])
                entry["worker"] = {"k": k, "tensors": errs, "update": upd,
                                   "loss": [float(losses[k]), loss_ref]}
                assert_tensors_close(errs, tol, "round 1 worker")
                # the change a few steps make, relative to its own size
                assert_tensors_close(upd, 5e-2, "round 1 worker update")
            worst = max(max(e["rel"], e["max"]) for e in entry.get("sampled", {}).values()) \
                if "sampled" in entry else None
            say(f"    loss rel <= {max(entry['loss_rel']):.2e}, norm rel <= "
                f"{max(entry['norm_rel'].values()):.2e}, sampled worst {worst}")
            log["rounds"].append(entry)
            del reps
    finally:
        record(f"full-size-{name}", log)
        unpack_ctx.close()
        run.close()
