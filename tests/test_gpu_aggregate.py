"""GPU parity of the parameter-server aggregation (Approach, Eq. 4, first
branch) against the oracle's pairwise tree: bit for bit."""
import numpy as np
import pytest

import oracle
import workload
from _parity import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def P():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2102_08550_amd
    return paper_2102_08550_amd


CASES = [(1, 1, 4), (1, 1000, 1000), (2, 4099, 4100), (3, 777, 780), (5, 10007, 10008),
         (8, 1 << 20, 1 << 20), (16, 65537, 65540), (32, 300001, 300004), (33, 4097, 4100),
         (64, 5003, 5004)]


@pytest.mark.parametrize("K,n,ld", CASES)
@pytest.mark.parametrize("bcast", [0, 1])
def test_aggregate_bitwise(P, K, n, ld, bcast):
    import torch
    say(f"aggregate K={K} n={n} ld={ld} broadcast={bcast}")
    rng = np.random.default_rng(K * 1000 + n)
    reps = rng.standard_normal((K, ld)).astype(np.float32)
    w = oracle.paper_weights(K)
    dr = torch.from_numpy(reps).cuda()
    dg = torch.full((n,), float("nan"), device="cuda")
    P.aggregate(dg, dr, w, K, n, ld, bool(bcast))
    torch.cuda.synchronize()
    expect = oracle.tree_aggregate([reps[k, :n] for k in range(K)], w)
    got = dg.cpu().numpy()
    assert np.array_equal(got.view(np.uint32), expect.view(np.uint32))
    back = dr.cpu().numpy()
    if bcast:
        assert np.array_equal(back[:, :n], np.broadcast_to(expect, (K, n)))
        assert np.array_equal(back[:, n:], reps[:, n:])
    else:
        assert np.array_equal(back, reps)


def test_aggregate_nonuniform_weights_bitwise(P):
    import torch
    rng = np.random.default_rng(5)
    for K in (3, 8, 20):
        n = 50001
        reps = rng.standard_normal((K, n + 3)).astype(np.float32)
        w = rng.uniform(-1, 1, K).astype(np.float32)
        dg = torch.empty(n, device="cuda")
        P.aggregate(dg, torch.from_numpy(reps).cuda(), w, K, n, n + 3)
        torch.cuda.synchronize()
        expect = oracle.tree_aggregate([reps[k, :n] for k in range(K)], w)
        assert np.array_equal(dg.cpu().numpy().view(np.uint32), expect.view(np.uint32))


def test_identical_replicas_identity(P):
    import torch
    n, ld = 100003, 100004
    x = np.random.default_rng(1).standard_normal(ld).astype(np.float32)
    for K in (1, 2, 4, 8, 16, 32, 64):
        dg = torch.empty(n, device="cuda")
        P.aggregate(dg, torch.from_numpy(np.tile(x, K)).cuda(), oracle.paper_weights(K), K, n, ld)
        torch.cuda.synchronize()
        assert np.array_equal(dg.cpu().numpy().view(np.uint32), x[:n].view(np.uint32))


def test_aggregate_rejects_bad_arguments(P):
    import torch
    dr = torch.zeros(4 * 1024, device="cuda")
    dg = torch.zeros(1024, device="cuda")
    w = oracle.paper_weights(4)
    bad = [dict(K=0), dict(K=65), dict(n=0), dict(ld=1022), dict(ld=1025)]
    for b in bad:
        args = dict(K=4, n=1024, ld=1024)
        args.update(b)
        with pytest.raises((P.OscarsError, ValueError)):
            ww = oracle.paper_weights(max(args["K"], 1))
            P.aggregate(dg, dr, ww, args["K"], args["n"], args["ld"])
    with pytest.raises(P.OscarsError) as ei:  # 4-byte aligned but not 16-byte aligned
        P.aggregate(dg[1:], dr, w, 4, 512, 1024)
    assert ei.value.status == P.E_INVALID
    with pytest.raises(P.OscarsError):  # global overlaps the replicas
        P.aggregate(dr, dr, w, 4, 1024, 1024)
    with pytest.raises(P.OscarsError):  # non-finite weight
        P.aggregate(dg, dr, np.array([0.25, np.nan, 0.25, 0.25], np.float32), 4, 1024, 1024)


@pytest.mark.parametrize("K,n,ld", [(1, 1, 4), (1, 1 << 20, 1 << 20), (3, 100003, 100004),
                                    (8, 54_440_960, 54_440_960), (64, 4097, 4100)])
def test_broadcast_copies_bit_for_bit(P, K, n, ld):
    """Every replica's first n elements become the global model; the padding
    between n and ld is left as it was."""
    import torch
    g = torch.from_numpy(np.random.default_rng(K).standard_normal(n).astype(np.float32)).cuda()
    reps = torch.full(((K - 1) * ld + n + (ld - n),), -7.0, device="cuda")
    P.broadcast(g, reps, K, n, ld)
    torch.cuda.synchronize()
    view = reps[: K * ld].view(K, ld)
    assert torch.equal(view[:, :n], g.unsqueeze(0).expand(K, n))
    if ld > n:
        assert torch.all(view[:, n:] == -7.0)


def test_broadcast_rejects_bad_arguments(P):
    import torch
    dr = torch.zeros(4 * 1024, device="cuda")
    dg = torch.zeros(1024, device="cuda")
    for K, n, ld in ((0, 1024, 1024), (65, 1024, 1024), (4, 0, 1024), (4, 1024, 1022),
                     (4, 1024, 1025)):
        with pytest.raises((P.OscarsError, ValueError)):
            P.broadcast(dg, dr, K, n, ld)
    with pytest.raises(P.OscarsError):
        P.broadcast(dg[1:], dr, 4, 512, 1024)  # not 16-byte aligned
    with pytest.raises(P.OscarsError):
        P.broadcast(dr, dr, 4, 1024, 1024)  # global overlaps the replicas
    torch.cuda.synchronize()
    assert torch.all(dr == 0.0)


def test_c4_full_size_sampled_100_rounds(P):
    """Aggregation stress workload at its full size: K = 32 replicas of 25.6M
    fp32, replicas = g + delta_k before each round, aggregate + broadcast, 100
    rounds.  The oracle follows one million sampled coordinates through all
    rounds (the average is coordinate-wise) and must agree bit for bit."""
    import torch
    cfg = workload.C4
    say("C4: generating 32 x 25.6M inputs")
    g0, delta = workload.gen_agg_vectors(cfg)
    stale = workload.gen_staleness(cfg)
    n, K = cfg.n_flat, cfg.K
    idx = np.sort(np.random.default_rng(0).choice(n, 1_000_000, replace=False))
    idx[-1] = n - 1
    og = g0[idx].copy()
    od = delta[:, idx].copy()
    G = torch.from_numpy(g0).cuda()
    D = torch.from_numpy(delta).cuda()
    del delta
    R = torch.empty_like(D)
    tidx = torch.from_numpy(idx).cuda()
    for r in range(cfg.rounds):
        w = P.paper_weights(K, stale[r])
        torch.add(G.unsqueeze(0), D, out=R)
        P.aggregate(G, R, w, K, n, n, True)
        og = oracle.tree_aggregate([og + od[k] for k in range(K)], oracle.paper_weights(K, stale[r]))
        got = G[tidx].cpu().numpy()
        assert np.array_equal(got.view(np.uint32), og.view(np.uint32)), f"round {r}"
        if r % 25 == 0:
            assert torch.equal(R[:, tidx], G[tidx].unsqueeze(0).expand(K, -1)), f"broadcast {r}"
        if r % 20 == 0:
            say(f"C4 round {r} ok")
    del R, D, G
    torch.cuda.empty_cache()
