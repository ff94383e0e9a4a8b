"""oscars_evaluate_noalloc (held-out evaluation for callers that cannot
allocate device memory) against oscars_evaluate through the C ABI: the same
summed loss and correct count, bit for bit, on two calls in a row -- the
second with fewer rows, so stale temporaries of the first call would show --
for a bf16 and an fp32 model; sizes above the limit are refused."""
import ctypes

import numpy as np
import pytest

import workload
from _parity import say

pytestmark = pytest.mark.gpu

CFGS = [
    workload.Config("noalloc-bf16", (264, 136, 72, 37), workload.BF16, K=2, n_rows=10, batch=96,
                    tau_rule="given", tau_given=(1, 1), seed=31),
    workload.Config("noalloc-fp32", (72, 264, 10), workload.FP32, K=1, n_rows=10, batch=200,
                    tau_rule="given", tau_given=(1,), seed=32),
]


@pytest.fixture(scope="module")
def P():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2102_08550_amd
    return paper_2102_08550_amd


def _dev(ds):
    import torch
    x = torch.from_numpy(np.ascontiguousarray(ds.x).view(np.int16)
                         if ds.dtype == workload.BF16 else ds.x).cuda()
    return x, torch.from_numpy(ds.y.astype(np.int32)).cuda()


@pytest.mark.parametrize("cfg", CFGS, ids=[c.name for c in CFGS])
def test_noalloc_evaluate_equals_evaluate(P, cfg):
    import torch
    say(f"noalloc evaluate {cfg.name}")
    ctx = P.Context(cfg.dims, P.BF16 if cfg.dtype == workload.BF16 else P.FP32, cfg.K, cfg.batch)
    try:
        params = torch.from_numpy(ctx.pack(workload.gen_init(cfg))).cuda()
        ev = workload.gen_eval_set(cfg, 5 * cfg.batch + 3)
        x, y = _dev(ev)
        for n in (5 * cfg.batch + 3, cfg.batch - 7):  # the second call smaller
            ref = ctx.evaluate(params, x, y, n)
            got = ctx.evaluate(params, x, y, n, noalloc=True)
            say(f"  n={n}: evaluate {ref}, noalloc {got}")
            assert np.float64(got[0]).view(np.uint64) == np.float64(ref[0]).view(np.uint64)
            assert got[1] == ref[1]
        # the limit, and the ordinary argument checks
        lib = P._lib()
        loss, hits = ctypes.c_double(0.0), ctypes.c_int64(0)
        for bad_n in (P.EVAL_NOALLOC_MAX_ROWS + 1, 0):
            st = lib.oscars_evaluate_noalloc(ctx._h, params.data_ptr(), x.data_ptr(),
                                             y.data_ptr(), bad_n, ctypes.byref(loss),
                                             ctypes.byref(hits))
            assert st == P.E_INVALID, (bad_n, st)
        with pytest.raises(P.OscarsError):
            ctx.evaluate(params[1:], x, y, 10, noalloc=True)  # not 16-byte aligned
    finally:
        ctx.close()
