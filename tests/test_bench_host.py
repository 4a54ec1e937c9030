"""Host-side logic of bench.py that needs no GPU: the one-GPU refusal, and the HBM-traffic figures
derived from rocprofv3 counter files (scaling by the calibration copy, per-launch averages, the
source digest that retires a figure when its kernel's sources change)."""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]


def _counters(path, counter, rows):
    with open(path, "w", newline="") as fh:
        wr = csv.DictWriter(fh, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        wr.writeheader()
        for name, value in rows:
            wr.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value})


def test_traffic_from_counter_files(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "hbm_traffic.json"))
    ev = "void tacg::(anonymous namespace)::ev_main<8, 2, false>(tacg::(anonymous namespace)::EvArgs)"
    hist = "void tacg::(anonymous namespace)::coact_hist_kernel<8, 1024>(tacg::(anonymous namespace)::CoactArgs)"
    red = "void tacg::(anonymous namespace)::coact_reduce_kernel<false, 4>(tacg::(anonymous namespace)::CoactArgs, ...)"
    copy = "__amd_rocclr_copyBuffer"
    # the 1 GiB calibration copy reads as 524,288 KiB (FETCH: scale 2) and 1,048,576 KiB (WRITE: scale 1);
    # a smaller copy of the run must not set the scale
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    _counters(fetch, "FETCH_SIZE", [(copy, 4.0), (copy, 524288.0), (ev, 100.0), (ev, 300.0), (hist, 10.0), (red, 1.0)])
    _counters(write, "WRITE_SIZE", [(copy, 1048576.0), (ev, 50.0), (hist, 2.0), (red, 3.0)])
    out = bench.write_traffic(str(fetch), str(write), "deepseek_v3")
    assert out["scale"] == {"FETCH_SIZE": 2.0, "WRITE_SIZE": 1.0}
    e = out["kernels"]["ev_main"]
    assert e["fetch_bytes"] == 200.0 * 1024 * 2          # mean of the two launches, scaled
    assert e["write_bytes"] == 50.0 * 1024
    c = out["kernels"]["coact_build"]                    # the two kernels of one build add up
    assert c["fetch_bytes"] == (10.0 + 1.0) * 1024 * 2
    assert c["write_bytes"] == (2.0 + 3.0) * 1024
    assert c["bytes_per_launch"] == c["fetch_bytes"] + c["write_bytes"]
    # the figure is reported for this workload and these sources only
    assert bench.measured_traffic("ev_main", "deepseek_v3") == e["bytes_per_launch"]
    assert bench.measured_traffic("ev_main", "qwen3_30b") is None
    rec = json.load(open(bench.TRAFFIC_FILE))
    rec["kernels"]["ev_main"]["source_sha256"] = "0" * 64
    json.dump(rec, open(bench.TRAFFIC_FILE, "w"))
    assert bench.measured_traffic("ev_main", "deepseek_v3") is None


def test_traffic_needs_the_calibration_copy(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "hbm_traffic.json"))
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    _counters(fetch, "FETCH_SIZE", [("void tacg::(anonymous namespace)::ev_main<8, 2, false>(x)", 1.0)])
    _counters(write, "WRITE_SIZE", [("__amd_rocclr_copyBuffer", 1048576.0)])
    with pytest.raises(SystemExit):
        bench.write_traffic(str(fetch), str(write), "deepseek_v3")
