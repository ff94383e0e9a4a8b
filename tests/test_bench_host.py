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

