"""bench.py's host logic without a GPU: the one-GPU rule, the counter bookkeeping that turns
rocprofv3 --pmc rows into bytes per E-step call, and the rule that a traffic figure is only
reported for the kernel source it was measured on."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def _pmc_csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, v) in enumerate(rows):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": name, "Counter_Value": v})


def _estep_rows(calls, logz_kib, other_kib):
    rows = []
    for c in range(calls):
        rows += [("k_prep_class(...)", 1.0), ("k_logz<128, true, false>(...)", logz_kib[c]),
                 ("k_stats_well<128, false>(...)", other_kib), ("at::native::fill(...)", 999.0)]
    return rows


def test_counter_per_call_skips_warmup_and_other_kernels(tmp_path):
    p = tmp_path / "c.csv"
    _pmc_csv(p, _estep_rows(4, [100.0, 200.0, 10.0, 30.0], 5.0))
    # per call: k_prep_class (1) + k_logz + k_stats_well (5); torch's fill is not an E-step kernel
    assert bench.counter_per_call(str(p), skip=2) == pytest.approx((1 + 10 + 5 + 1 + 30 + 5) / 2)
    assert bench.counter_per_call(str(p), ("k_logz",), skip=2) == pytest.approx(20.0)
    assert bench.counter_per_call(str(p), ("k_logz",), skip=0) == pytest.approx(85.0)


def test_write_traffic_scales_by_the_copy_and_records_the_source(tmp_path, monkeypatch):
    os.makedirs(tmp_path / "profiles")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    # the copy reads COPY_BYTES, FETCH_SIZE sees half of it, WRITE_SIZE all of it (KiB)
    cb = bench.COPY_BYTES / 1024.0
    _pmc_csv(tmp_path / "fc.csv", [("__amd_rocclr_copyBuffer", cb / 2)])
    _pmc_csv(tmp_path / "wc.csv", [("__amd_rocclr_copyBuffer", cb)])
    _pmc_csv(tmp_path / "f.csv", _estep_rows(3, [1000.0, 1000.0, 1000.0], 50.0))
    _pmc_csv(tmp_path / "w.csv", _estep_rows(3, [10.0, 10.0, 10.0], 0.0))
    monkeypatch.setattr(bench, "source_digest", lambda: "abc")
    bench.write_traffic("unit", str(tmp_path / "f.csv"), str(tmp_path / "w.csv"),
                        str(tmp_path / "fc.csv"), str(tmp_path / "wc.csv"), skip=1)
    t = json.load(open(tmp_path / "profiles" / "estep_traffic_unit.json"))
    assert t["fetch_scale"] == pytest.approx(2.0) and t["write_scale"] == pytest.approx(1.0)
    assert t["logz_fetch_bytes"] == pytest.approx(2 * 1000 * 1024)
    assert t["logz_bytes_per_launch"] == pytest.approx(2 * 1000 * 1024 + 10 * 1024)
    assert t["bytes_per_call"] == pytest.approx(2 * 1051 * 1024 + 11 * 1024)
    assert t["source_sha256"] == "abc"
    # reported only while the kernel source is the one the counters ran on
    assert bench.measured_traffic("unit") == pytest.approx(t["logz_bytes_per_launch"])
    monkeypatch.setattr(bench, "source_digest", lambda: "changed")
    assert bench.measured_traffic("unit") is None
