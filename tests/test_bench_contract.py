"""Host-side parts of bench.py (no GPU): the one-GPU refusal, the rule that
HBM traffic is reported only for the kernel source it was measured on, and
the split of a rocprofv3 kernel trace by the dispatch windows the JSON line
records."""
import csv
import hashlib
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
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_traffic_only_for_the_measured_source(tmp_path, monkeypatch):
    src = tmp_path / "kernel.hip"
    src.write_text("// a kernel\n")
    sha = hashlib.sha256(src.read_bytes()).hexdigest()
    monkeypatch.setattr(bench, "TRAFFIC", {"cX": {"source": str(src), "sha256": sha, "fetch_bytes": 1000.0,
                                                  "write_bytes": 24.0, "kv_bytes": 1000}})
    r = bench.roofline("cX", "k", 4000.0, 1000)
    assert r["traffic"] == 1024 and r["traffic_per_kv_byte"] == 1.024
    assert r["frac"] == 0.5 and r["peak"] == 8000.0 and r["bound"] == "hbm"
    src.write_text("// a kernel, changed\n")
    r = bench.roofline("cX", "k", 4000.0, 1000)
    assert r["traffic"] is None and "traffic_per_kv_byte" not in r
    assert bench.roofline("other", "k", 4000.0, 1000)["traffic"] is None


def test_traffic_table_sources_exist():
    for key, t in bench.TRAFFIC.items():
        assert os.path.isfile(os.path.join(ROOT, t["source"])), key
        assert len(t["sha256"]) == 64 and t["kv_bytes"] > 0, key


def _trace(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Dispatch_Id", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        for r in rows:
            w.writerow(r)


def test_trace_summary_splits_by_dispatch_window(tmp_path, capsys):
    # dispatch order: 2 pass-1-alone launches, then an unrelated kernel, then
    # 3 step launches (one of them the flat-split instantiation): the window
    # [first, count, kernel] picks by kernel name in dispatch order
    rows, t, d = [], 0, 1
    def launch(name, us):
        nonlocal t, d
        rows.append({"Kernel_Name": name, "Dispatch_Id": d, "Start_Timestamp": t, "End_Timestamp": t + int(us * 1000)})
        t += int(us * 1000) + 500
        d += 1
    launch("void gqa_attend_kernel<8, false>(AttendParams)", 100.0)
    launch("void gqa_attend_kernel<8, false>(AttendParams)", 102.0)
    launch("at::native::reduce_kernel<...>", 50.0)
    launch("void gqa_step_kernel<8, false>(AttendParams, StepTail)", 110.0)
    launch("void gqa_step_kernel<8, true>(AttendParams, StepTail)", 112.0)
    launch("void gqa_step_kernel<8, false>(AttendParams, StepTail)", 114.0)
    os.makedirs(tmp_path / "run")
    _trace(tmp_path / "run" / "run_kernel_trace.csv", rows)
    line = {"metric": "m", "value": 1.0,
            "config": {"kv_bytes_per_step": 1_000_000_000},
            "breakdown_us": {"step": 111.5, "pass1_kernel": 101.5, "pass1_kv_bytes": 1_000_000_000},
            "roofline": {"kv_bytes_per_launch": 1_000_000_000},
            "dispatch_window": {"kernel": "gqa_step_kernel<8>",
                                "timed_steps": [1, 2, "gqa_step_kernel<8>"],
                                "pass1_alone": [0, 2, "gqa_attend_kernel<8>"]}}
    js = tmp_path / "b.json"
    js.write_text("progress\n" + json.dumps(line) + "\n")
    bench.trace_summary(str(tmp_path), str(js))
    out = capsys.readouterr().out
    rows_out = {ln.split("|")[3].strip(): [c.strip() for c in ln.split("|")] for ln in out.splitlines()
                if ln.startswith("| headline")}
    step = rows_out["timed_steps"]
    assert step[2] == "gqa_step_kernel<8>" and step[4] == "2"
    assert float(step[5]) == pytest.approx(113.0) and float(step[6]) == 112.0 and float(step[7]) == 114.0
    assert float(step[11]) == 111.5                      # bench.py's own time of the part, beside it
    p1 = rows_out["pass1_alone"]
    assert float(p1[5]) == pytest.approx(101.0) and p1[4] == "2"
    assert float(p1[8]) == 1000.0                        # KV MB per launch
    assert float(p1[9]) == pytest.approx(1e9 / 101e-6 / 1e12, abs=0.005)   # TB/s at the mean, 2 decimals
