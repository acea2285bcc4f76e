"""Host-side logic of bench.py (no GPU): the one-GPU guard, the copy-calibrated traffic
summary of two rocprofv3 counter files, and the staleness check of stored traffic."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"]


def _counter_csv(path, counter, rows):
    """rows: (dispatch id, kernel name, per-XCD values) -> a counter file as rocprofv3 writes it."""
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for did, name, values in rows:
            for v in values:  # several records per dispatch are summed
                w.writerow({"Dispatch_Id": did, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": v})


def test_traffic_summary_scales_each_counter_by_the_copy_kernel(tmp_path):
    copy = "void at::native::neg_kernel(float)"
    dkv = "void sra::sra_dkv_kernel<128, true>(sra::BwdArgs)"
    delta = "void sra::sra_delta_kernel<128>(sra::DeltaArgs, int)"
    # copy of 64 MiB: fetch reads a quarter of the bytes, write half (as on MI355X)
    fetch = tmp_path / "fetch.csv"
    write = tmp_path / "write.csv"
    _counter_csv(fetch, "FETCH_SIZE", [(1, copy, [8192.0, 8192.0]), (2, dkv, [1000.0, 500.0]),
                                       (3, delta, [100.0]), (4, delta, [300.0]),
                                       (5, "void other_kernel()", [7.0])])
    _counter_csv(write, "WRITE_SIZE", [(1, copy, [32768.0]), (2, dkv, [10.0]), (3, delta, [4.0]), (4, delta, [6.0])])
    out = tmp_path / "traffic.json"
    bench._pmc_summary(str(fetch), str(write), 64, "720p", str(out))
    data = json.loads(out.read_text())
    cal = data["calibration"]
    assert cal["fetch_scale"] == pytest.approx(4.0) and cal["write_scale"] == pytest.approx(2.0)
    k = data["kernels"]["dkdv"]
    assert k["fetch_kib_raw"] == 1500.0 and k["fetch_bytes"] == round(1500.0 * 4 * 1024)
    assert k["write_bytes"] == round(10.0 * 2 * 1024) and k["dispatches"] == 1
    d = data["kernels"]["delta"]  # mean over its two dispatches
    assert d["dispatches"] == 2 and d["fetch_kib_raw"] == 200.0 and d["write_kib_raw"] == 5.0
    assert set(data["kernels"]) == {"dkdv", "delta"}


def test_traffic_summary_needs_the_copy_kernel(tmp_path):
    f = tmp_path / "f.csv"
    _counter_csv(f, "FETCH_SIZE", [(2, "void sra::sra_fwd_kernel<128>(sra::FwdArgs)", [1.0])])
    with pytest.raises(SystemExit):
        bench._pmc_summary(str(f), str(f), 64, "720p", str(tmp_path / "o.json"))


def test_stored_traffic_is_dropped_when_the_kernel_source_changes(tmp_path, monkeypatch):
    h = bench._kernel_source_hash("dkdv")
    stored = {"workload": "720p", "kernels": {"dkdv": {"source_hash": h, "fetch_bytes": 10, "write_bytes": 5}}}
    p = tmp_path / "t.json"
    p.write_text(json.dumps(stored))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(p))
    assert bench._stored_traffic("dkdv", "720p") == 15
    assert bench._stored_traffic("dkdv", "varlen") is None  # another workload's counters
    stored["kernels"]["dkdv"]["source_hash"] = "0" * 16
    p.write_text(json.dumps(stored))
    assert bench._stored_traffic("dkdv", "720p") is None


def test_cpu_baseline_reports_fp32_legs_and_an_extrapolated_layer():
    """The CPU-oracle leg of the benchmark on a small layer: float32 forward rows (float64
    beside), dQ rows, the full forward and backward of a frame slice and the tiny workload,
    seconds per layer extrapolated from them, and the host's CPU description."""
    import torch

    from paper_2606_13872_amd import sra
    from sra_inputs import SampleGeom, Workload, make_inputs

    w = Workload("small", [SampleGeom(3, 8, 8, 3, 8, 8)], 2, 64, 5, False)
    x = make_inputs(w.samples, w.heads, w.head_dim, w.seed)
    fwd, _ = sra.useful_flops(w.samples, w.heads, w.head_dim)
    out = bench._cpu_baseline(x, w, 32, torch, fwd // (4 * w.head_dim))
    assert out["kind"] == "oracle" and out["unit"] == "TFLOP/s" and out["value"] > 0
    assert out["cores"] >= 1 and out["nproc"] >= 1 and isinstance(out["cpu_model"], str)
    legs = out["legs"]
    assert legs["fwd"]["dtype"] == "float32" and legs["fwd_float64"]["dtype"] == "float64"
    assert legs["fwd"]["visible_pairs"] == 32 * (192 + 192) + 32 * 64
    for k in ("dq", "slice", "tiny"):
        assert k in legs
    s = out["seconds_per_layer_extrapolated"]
    assert s["step"] == pytest.approx(s["fwd"] + s["bwd"], abs=0.11)
