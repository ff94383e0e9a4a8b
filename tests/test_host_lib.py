"""CPU tests of the C-ABI library: it loads, exports every declared entry
point, and its host-only parts (Algorithm 1, shards, sampler, weights) agree
bit for bit with the oracle.  No GPU work is started here."""
import ctypes
import os
import random
import re
import subprocess
import sys

import numpy as np
import pytest

import oracle
import workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "oscars.h")
LIBDIR = os.path.join(ROOT, "paper_2102_08550_amd", "_lib")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(oscars_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(os.path.join(LIBDIR, "liboscars.so"))
    names = _declared()
    assert len(names) >= 18
    for n in names:
        assert hasattr(lib, n), n


def test_binding_covers_header():
    import paper_2102_08550_amd as P
    assert set(_declared()) == set(P._SIGS)


@pytest.fixture(scope="module")
def P():
    import paper_2102_08550_amd
    return paper_2102_08550_amd


def test_context_knobs_reject_bad_arguments(P):
    """Tiling, backward mode and the tuning count belong to a context: a null
    context or output, or a value outside its range, is refused with
    E_INVALID before anything is touched (no GPU work)."""
    lib = P._lib()
    for t in (P.TILING_AUTO, len(P.TILINGS), -1):
        assert lib.oscars_set_gemm_tiling(None, t) == P.E_INVALID
    for m in (P.BACKWARD_AUTO, len(P.BACKWARDS), -1):
        assert lib.oscars_set_backward(None, m) == P.E_INVALID
    n = P._i32(0)
    assert lib.oscars_tuning_pending(None, P.ctypes.byref(n)) == P.E_INVALID
    assert lib.oscars_tuning_pending(None, None) == P.E_INVALID


def test_load_balance_matches_oracle(P):
    rnd = random.Random(3)
    for _ in range(400):
        N = rnd.randint(1, 9)
        t = [rnd.randint(1, 30) for _ in range(N)]
        M = rnd.randint(1, 10)
        try:
            expect = oracle.load_balance(t, M)
        except oracle.InfeasibleBarrier:
            with pytest.raises(P.OscarsError) as ei:
                P.load_balance(t, M)
            assert ei.value.status == P.E_INFEASIBLE
            continue
        assert P.load_balance(t, M) == expect
    for cfg in (workload.C2, workload.C5):
        t = workload.speeds_to_t_iter(cfg.speeds)
        assert P.load_balance(t, cfg.M) == oracle.load_balance(t, cfg.M)


def test_load_balance_bad_args(P):
    for t, M in (([], 3), ([0, 2], 3), ([1, 2], 0), ([-1], 2)):
        with pytest.raises(P.OscarsError) as ei:
            P.load_balance(t, M)
        assert ei.value.status == P.E_INVALID


def test_plan_tau_matches_oracle(P):
    """Quantized measured times and the resulting plan: bit-exact with the oracle."""
    rnd = random.Random(5)
    for _ in range(400):
        N = rnd.randint(1, 9)
        t = [rnd.uniform(0.05, 9.0) * 10 ** rnd.randint(-3, 3) for _ in range(N)]
        R = rnd.randint(1, 40)
        M = rnd.randint(1, 12)
        ticks = oracle.quantize_iteration_times(t, R)
        if max(ticks) > 2**30:  # above the library's tick limit: rejected, not scanned
            with pytest.raises(P.OscarsError) as ei:
                P.plan_tau(t, R, M)
            assert ei.value.status == P.E_INVALID
            continue
        try:
            expect = oracle.plan_from_measured(t, R, M)
        except oracle.InfeasibleBarrier:
            with pytest.raises(P.OscarsError) as ei:
                P.plan_tau(t, R, M)
            assert ei.value.status == P.E_INFEASIBLE
            continue
        assert P.plan_tau(t, R, M) == (expect[0], expect[1], expect[2])
    # halves round up on both sides
    assert P.plan_tau([2.0, 3.25, 3.1, 9.0], 4, 8)[0] == [4, 7, 6, 18]


def test_plan_tau_bad_args(P):
    for t, R, M in (([], 2, 3), ([1.0, 0.0], 2, 3), ([1.0, float("nan")], 2, 3),
                    ([1.0, float("inf")], 2, 3), ([1.0], 0, 3), ([1.0], 4097, 3),
                    ([1.0], 2, 0), ([1.0, 1e12], 4096, 3)):
        with pytest.raises(P.OscarsError) as ei:
            P.plan_tau(t, R, M)
        assert ei.value.status == P.E_INVALID, (t, R, M)


def test_shard_offsets_match_oracle(P):
    for N, K in [(8192, 4), (60000, 8), (50000, 16), (200000, 8), (23, 4), (5, 7), (0, 3),
                 (2**40 + 3, 64)]:
        assert P.shard_offsets(N, K) == oracle.shard_offsets(N, K)


def test_paper_weights(P):
    for K in (1, 3, 8, 32, 64):
        w = P.paper_weights(K, staleness=list(range(K)))
        assert np.array_equal(w, oracle.paper_weights(K))
        assert np.array_equal(w, P.paper_weights(K))


@pytest.mark.parametrize("cfg", [workload.C1, workload.C2, workload.C3, workload.C5],
                         ids=lambda c: c.name)
def test_sampler_bit_exact_on_workload_shards(P, cfg):
    seed = workload.sampler_seed(cfg)
    off = oracle.shard_offsets(cfg.n_rows, cfg.K)
    cache = {}
    for k in (0, cfg.K // 2, cfg.K - 1):
        n_k = off[k + 1] - off[k]
        # steps around the first two epoch boundaries and the start
        first_cross = n_k // cfg.batch
        for s0 in (0, max(first_cross - 1, 0), max(2 * n_k // cfg.batch - 1, 0)):
            got = P.sample_indices(cfg.n_rows, off, seed, k, s0, 3, cfg.batch)
            exp = [oracle.batch_rows(seed, off, k, s0 + j, cfg.batch, cache) for j in range(3)]
            assert np.array_equal(got, np.array(exp)), (k, s0)


def test_sampler_bad_args(P):
    off = [0, 3, 3, 9]  # worker 1 has an empty shard
    with pytest.raises(P.OscarsError):
        P.sample_indices(9, off, 1, 1, 0, 1, 2)
    with pytest.raises(P.OscarsError):
        P.sample_indices(9, [0, 3, 6, 9], 1, 3, 0, 1, 2)  # k out of range


def test_host_logic_under_sanitizers():
    """The host-only build with ASan + UBSan runs Algorithm 1 and the sampler
    without a report (child process with the ASan runtime preloaded)."""
    san = os.path.join(LIBDIR, "liboscars_host_san.so")
    if not os.path.exists(san):
        pytest.skip("sanitizer build not available")
    asan = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("libasan not found")
    code = r"""
import ctypes, sys
import numpy as np
lib = ctypes.CDLL(sys.argv[1])
P = ctypes.POINTER
t = np.array([24, 24, 12, 12, 8, 6, 4, 3], np.int64); tau = np.zeros(8, np.int32)
T = ctypes.c_int64(0)
assert lib.oscars_load_balance(t.ctypes.data_as(P(ctypes.c_int64)), 8, ctypes.c_int64(8),
                               ctypes.byref(T), tau.ctypes.data_as(P(ctypes.c_int32))) == 0
assert T.value == 24 and tau.tolist() == [1, 1, 2, 2, 3, 4, 6, 8]
tm = np.array([2.4, 2.4, 1.2, 1.2, 0.8, 0.6, 0.4, 0.3]); ticks = np.zeros(8, np.int64)
assert lib.oscars_plan_tau(tm.ctypes.data_as(P(ctypes.c_double)), 8, 3, ctypes.c_int64(8),
                           ticks.ctypes.data_as(P(ctypes.c_int64)), ctypes.byref(T),
                           tau.ctypes.data_as(P(ctypes.c_int32))) == 0
assert ticks.tolist() == [24, 24, 12, 12, 8, 6, 4, 3] and tau.tolist() == [1, 1, 2, 2, 3, 4, 6, 8]
class S(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("y", ctypes.c_void_p), ("n_rows", ctypes.c_int64),
                ("offsets", P(ctypes.c_int64)), ("seed", ctypes.c_uint64)]
off = np.zeros(9, np.int64)
assert lib.oscars_shard_offsets(ctypes.c_int64(60000), 8, off.ctypes.data_as(P(ctypes.c_int64))) == 0
s = S(None, None, 60000, off.ctypes.data_as(P(ctypes.c_int64)), 12345)
rows = np.zeros((130, 64), np.int64)
for k in range(8):
    assert lib.oscars_sample_indices(ctypes.byref(s), 8, k, ctypes.c_int64(100), 130, 64,
                                     rows.ctypes.data_as(P(ctypes.c_int64))) == 0
    assert rows.min() >= off[k] and rows.max() < off[k + 1]
print("sanitized-ok")
"""
    env = dict(os.environ, LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-c", code, san], capture_output=True, text=True, env=env,
                       timeout=300)
    assert r.returncode == 0 and "sanitized-ok" in r.stdout, r.stdout + r.stderr
