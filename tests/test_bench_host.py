"""bench.py host logic on the CPU: the multi-GPU request is refused before any
GPU work, traffic figures are used only while the kernel sources and launch
shape they were measured on are unchanged, and the bound arithmetic."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr and res.stdout == ""


def test_kernel_family_names():
    assert bench.kernel_family("split_row_kernel<rowsm::F32, rowsm::F32, 4, 16, 0, false>") \
        == "split_row"
    assert bench.kernel_family("bwd_split_kernel<rowsm::F32, rowsm::F32, 4, 8>") == "bwd"
    assert bench.kernel_family("group_top2_kernel<rowsm::F32, rowsm::F32, 4, 8, 4>") \
        == "group_top2"
    for fam in bench.KERNEL_SOURCES:
        assert len(bench.kernel_source_hash(fam)) == 16


def test_measured_traffic_only_for_unchanged_sources(tmp_path, monkeypatch):
    kern = "small_row_kernel<rowsm::BF16, rowsm::BF16, 8, 8, 4, 0>"
    launch = "small vw=8 ... grid=2048"
    entry = {"kernel": kern, "launch": launch, "hbm_bytes_per_launch": 123.0,
             "source_hash": bench.kernel_source_hash("small_row")}
    p = tmp_path / "traffic.json"
    p.write_text(json.dumps({"launches": {"w": entry}}))
    monkeypatch.setattr(bench, "PROFILE_COUNTERS", str(p))
    assert bench.measured_traffic("w", launch) == 123.0
    assert bench.measured_traffic("w", launch + " other") is None   # launch shape changed
    assert bench.measured_traffic("missing", launch) is None
    entry["source_hash"] = "0" * 16                                   # sources changed
    p.write_text(json.dumps({"launches": {"w": entry}}))
    assert bench.measured_traffic("w", launch) is None
    monkeypatch.setattr(bench, "PROFILE_COUNTERS", str(tmp_path / "absent.json"))
    assert bench.measured_traffic("w", launch) is None


def test_committed_traffic_table_is_well_formed():
    with open(bench.PROFILE_COUNTERS) as f:
        prof = json.load(f)
    assert 1.9 < prof["fetch_scale"] < 2.1 and 0.9 < prof["write_scale"] < 1.1
    for key, ent in prof["launches"].items():
        assert bench.kernel_family(ent["kernel"]) in bench.KERNEL_SOURCES, key
        assert ent["hbm_bytes_per_launch"] == pytest.approx(ent["fetch_bytes"] +
                                                            ent["write_bytes"])
        # every input byte fetched about once and every output byte written once
        assert 0.99 < ent["fetch_over_input_bytes"] < 1.05, key
        assert 0.99 < ent["write_over_output_bytes"] < 1.02, key


def test_mix_bound():
    r, w = bench.MEASURED_READ_GBS, bench.MEASURED_WRITE_GBS
    assert bench.mix_bound_gbs(1.0, 0.0) == pytest.approx(r)
    assert bench.mix_bound_gbs(0.0, 1.0) == pytest.approx(w)
    b = bench.mix_bound_gbs(1.0, 1.0)
    assert min(r, w) < b < max(r, w)
    assert b == pytest.approx(2.0 / (1.0 / r + 1.0 / w))
    assert set(bench.TARGET_FRAC) <= set(__import__(
        "paper_2607_23089_amd.workloads", fromlist=["REGIMES"]).REGIMES)
