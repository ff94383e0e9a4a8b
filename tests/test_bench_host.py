"""Host-side logic of bench.py (no GPU): the HBM traffic it reports comes
from the committed counter summary only while that summary matches the
kernel source."""
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _write(path, sha, ratio=1.25):
    json.dump({"c5": {"gemm_bwd_fused": {"kernels_sha256_16": sha, "ratio": ratio}}},
              open(path, "w"))


def test_traffic_follows_the_committed_ratio_for_the_current_source(tmp_path, monkeypatch):
    p = tmp_path / "pmc.json"
    _write(p, bench.kernel_source_hash())
    monkeypatch.setattr(bench, "PMC_FILE", str(p))
    assert bench.pmc_traffic("gemm_bwd_fused", "c5", 1000.0) == pytest.approx(1250.0)
    # another workload or kernel has no entry
    assert bench.pmc_traffic("gemm_bwd_fused", "c4", 1000.0) is None
    assert bench.pmc_traffic("gemm_fwd", "c5", 1000.0) is None


def test_traffic_is_null_once_the_kernels_changed(tmp_path, monkeypatch):
    p = tmp_path / "pmc.json"
    _write(p, "0000000000000000")
    monkeypatch.setattr(bench, "PMC_FILE", str(p))
    assert bench.pmc_traffic("gemm_bwd_fused", "c5", 1000.0) is None
    monkeypatch.setattr(bench, "PMC_FILE", str(tmp_path / "missing.json"))
    assert bench.pmc_traffic("gemm_bwd_fused", "c5", 1000.0) is None



def test_traffic_needs_the_same_launch_mix(tmp_path, monkeypatch):
    """A summary that records the backward path per layer and replica count
    applies only to runs that took the same paths."""
    p = tmp_path / "pmc.json"
    mix = {"l2": {"8": "fused", "1": "separate"}}
    json.dump({"c5": {"gemm_bwd_fused": {"kernels_sha256_16": bench.kernel_source_hash(),
                                         "ratio": 1.1, "backward_mix": mix}}}, open(p, "w"))
    monkeypatch.setattr(bench, "PMC_FILE", str(p))
    assert bench.pmc_traffic("gemm_bwd_fused", "c5", 1000.0, mix) == pytest.approx(1100.0)
    other = {"l2": {"8": "fused", "1": "fused"}}
    assert bench.pmc_traffic("gemm_bwd_fused", "c5", 1000.0, other) is None


def test_traffic_accepts_a_mix_of_nearly_the_same_bytes(tmp_path, monkeypatch):
    p = tmp_path / "pmc.json"
    theirs = {"l2": {"1": "fused"}}
    json.dump({"c5": {"gemm_bwd_fused": {"kernels_sha256_16": bench.kernel_source_hash(),
                                         "ratio": 1.1, "backward_mix": theirs}}}, open(p, "w"))
    monkeypatch.setattr(bench, "PMC_FILE", str(p))
    ours = {"l2": {"1": "separate"}}
    close = lambda m: 1000.0 if m == ours else 1020.0  # noqa: E731
    far = lambda m: 1000.0 if m == ours else 1200.0  # noqa: E731
    assert bench.pmc_traffic("gemm_bwd_fused", "c5", 500.0, ours, close) == pytest.approx(550.0)
    assert bench.pmc_traffic("gemm_bwd_fused", "c5", 500.0, ours, far) is None
