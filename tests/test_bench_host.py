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


def test_source_digest_follows_code_not_comments():
    """The traffic record's source digest changes with the code and not with comments or layout."""
    a = "int f(int x) {  // doubles\n  return 2 * x; /* a\n block */ }\n"
    assert bench.code_text(a) == bench.code_text("int f(int x) {\n\n return 2 * x; }")
    assert bench.code_text(a) != bench.code_text("int f(int x) { return 3 * x; }")
    assert bench.code_text("a = b; // x\nc = d;") == "a = b; c = d;"


def test_traffic_needs_the_calibration_copy(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "hbm_traffic.json"))
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    _counters(fetch, "FETCH_SIZE", [("void tacg::(anonymous namespace)::ev_main<8, 2, false>(x)", 1.0)])
    _counters(write, "WRITE_SIZE", [("__amd_rocclr_copyBuffer", 1048576.0)])
    with pytest.raises(SystemExit):
        bench.write_traffic(str(fetch), str(write), "deepseek_v3")


def test_single_thread_oracle_record():
    """The one-thread oracle figure of a preset: whole grouping trace and one placement, on one
    thread, with the trace's digest; the oracle's thread count is restored afterwards."""
    import oracle
    from paper_2606_01007_amd import synth

    oracle.build()
    before = oracle.num_threads()
    rec = bench.single_thread_oracle("tiny", device="cpu")
    assert oracle.num_threads() == before
    assert rec["cores"] == 1 and rec["err"] == 0
    assert rec["coact_value"] > 0 and rec["scoring_value"] > 0
    w = synth.make_workload("tiny")
    assert rec["trace_sha256"] == synth.trace_digest(w.trace_group)
    assert "6144 tokens x 2 layers" in rec["sample"]


def test_workload_seeds_are_the_generators_seeds():
    from paper_2606_01007_amd import synth

    s = synth.workload_seeds(synth.CONFIGS["qwen15"])
    assert s == {"logits_and_grouping_trace": 103, "serving_trace": 103, "placements_0": 1103,
                 "secondaries_0": 2103, "placements_1": 2103, "secondaries_1": 4103}
    s = synth.workload_seeds(synth.CONFIGS["deepseek_v3"])
    assert s["serving_trace"] == 205 and s["placements_0"] == 1105
    # the recorded seeds regenerate the recorded placements
    w = synth.make_workload("tiny")
    p = synth.random_placements(16, 2, 8, 4, 2, synth.workload_seeds(synth.CONFIGS["tiny"])["placements_0"])
    assert (p == w.placement_sets[0]["primary"]).all()
