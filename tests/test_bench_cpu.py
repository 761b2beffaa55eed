"""CPU tests of bench.py's host logic: the one-GPU contract and the HBM-traffic
calibration from rocprofv3 counter files (synthetic files here; no GPU is touched)."""
import csv
import importlib.util
import json
import os
import subprocess
import sys

import pytest

from conftest import ROOT


def load_bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def write_counters(path, counter, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for d, k, v in rows:
            w.writerow({"Dispatch_Id": d, "Kernel_Name": k, "Counter_Name": counter, "Counter_Value": v})


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_calibration(tmp_path, monkeypatch):
    """Each counter is scaled by what it reads for the calibration copy (4*K*N bytes each
    way, K = 3072), and only sparse-kernel dispatches before the copy count."""
    bench = load_bench()
    monkeypatch.setattr(bench, "traffic_file", lambda layer="w0": str(tmp_path / "traffic.json"))
    N = 4096
    copy_kib = 4 * 3072 * N / 1024            # 49152 KiB each way
    spmm = "void sdnn::spmm_panel_kernel<4, 1>(...)"
    neg = "void at::native::elementwise_kernel<128, 4, neg_kernel>(...)"
    fetch, write = tmp_path / "fetch.csv", tmp_path / "write.csv"
    # FETCH_SIZE counts half the copy's bytes (factor 2); WRITE_SIZE counts them exactly
    write_counters(fetch, "FETCH_SIZE", [(1, spmm, 1000.0), (2, spmm, 1100.0), (3, spmm, 1200.0),
                                         (4, neg, copy_kib / 2), (5, spmm, 9999.0)])
    write_counters(write, "WRITE_SIZE", [(1, spmm, 300.0), (2, spmm, 300.0), (3, spmm, 300.0),
                                         (4, neg, copy_kib), (5, spmm, 9999.0)])
    bench.summarize_pmc(str(fetch), str(write), 3072, N)
    out = json.load(open(tmp_path / "traffic.json"))
    assert out["kernel_hash"] == bench.kernel_hash()
    assert out["fetch_launches"] == 3 and out["write_launches"] == 3
    assert out["fetch_calibration_factor"] == pytest.approx(2.0)
    assert out["write_calibration_factor"] == pytest.approx(1.0)
    assert out["fetch_bytes_per_launch"] == pytest.approx(1100.0 * 1024 * 2)
    assert out["write_bytes_per_launch"] == pytest.approx(300.0 * 1024)
    assert out["bytes_per_launch"] == pytest.approx(1100.0 * 2048 + 300.0 * 1024)


def test_traffic_is_reported_only_for_the_profiled_sources(tmp_path, monkeypatch):
    bench = load_bench()
    path = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "traffic_file", lambda layer="w0": str(path))
    json.dump({"kernel_hash": "0" * 16, "bytes_per_launch": 123.0}, open(path, "w"))
    assert bench.measured_traffic() is None
    json.dump({"kernel_hash": bench.kernel_hash(), "bytes_per_launch": 123.0}, open(path, "w"))
    assert bench.measured_traffic() == 123.0

