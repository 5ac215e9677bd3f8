"""Host logic of rocprof_summary.py on small synthetic rocprofv3 CSV files:
the overlap fraction of the copy stream, the calibrated traffic record and
the mean over a window of one kernel's launches."""

import csv
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TOOL = os.path.join(ROOT, "rocprof_summary.py")

TRACE_FIELDS = ["Kind", "Stream_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp", "Grid_Size_X"]


def write_trace(path, rows):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "x_kernel_trace.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=TRACE_FIELDS)
        w.writeheader()
        for stream, name, a, b, grid in rows:
            w.writerow({"Kind": "KERNEL_DISPATCH", "Stream_Id": stream, "Kernel_Name": name,
                        "Start_Timestamp": a, "End_Timestamp": b, "Grid_Size_X": grid})


def run(*args):
    return subprocess.run([sys.executable, TOOL, *args], capture_output=True, text=True, check=True).stdout


def test_overlap_fraction(tmp_path):
    # copy 1 on stream 1: [0, 100 us], compute covers [20, 50] and [40, 90] -> 70%
    # copy 2: [200, 300 us], compute [150, 400] -> 100%
    us = 1000
    write_trace(str(tmp_path), [
        (1, "__amd_rocclr_copyBuffer", 0, 100 * us, 4096),
        (0, "void fs::gemm<0>(int)", 20 * us, 50 * us, 65536),
        (0, "void fs::gemm<1>(int)", 40 * us, 90 * us, 65536),
        (1, "__amd_rocclr_copyBuffer", 200 * us, 300 * us, 4096),
        (0, "void fs::combine(int)", 150 * us, 400 * us, 4096),
        (0, "__amd_rocclr_copyBuffer", 500 * us, 502 * us, 512),   # small setup copy elsewhere
    ])
    out = run(str(tmp_path), "--overlap", "--min-us", "10")
    assert "copy stream 1: 2 copies" in out
    assert "| 2 | 100.0 | 85.0% | 70.0% | 100.0% | 15.0 |" in out
    out = run(str(tmp_path), "--overlap", "--min-us", "10", "--skip", "1")
    assert "| 1 | 100.0 | 100.0% | 100.0% | 100.0% | 0.0 |" in out


def test_traffic_record(tmp_path):
    trace, fetch, write = (str(tmp_path / n) for n in ("trace", "fetch", "write"))
    write_trace(trace, [(0, "void fs::(anonymous namespace)::gemm_x<0, 128>(int)", 0, 10, 65536)])
    for d, counter, gemm_kib, copy_kib in ((fetch, "FETCH_SIZE", 1000, 512), (write, "WRITE_SIZE", 300, 1024)):
        os.makedirs(d)
        with open(os.path.join(d, "x_counter_collection.csv"), "w", newline="") as f:
            w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"])
            w.writeheader()
            w.writerow({"Kernel_Name": "void fs::(anonymous namespace)::gemm_x<0, 128>(int)",
                        "Grid_Size": 65536, "Counter_Name": counter, "Counter_Value": gemm_kib})
            w.writerow({"Kernel_Name": "__amd_rocclr_copyBuffer", "Grid_Size": 4096,
                        "Counter_Name": counter, "Counter_Value": copy_kib})
    src = tmp_path / "src.hip"
    src.write_text("kernel source\n")
    out_json = str(tmp_path / "rec.json")
    run(trace, "--fetch", fetch, "--write", write, "--copy-bytes", str(1024 * 1024),
        "--traffic-json", out_json, "--kernel", "gemm_x<0, 128>", "--workload", "w",
        "--source", str(src), "--command", "cmd")
    rec = json.load(open(out_json))
    # the 1 MiB copy reads 512 KiB of FETCH (scale 2) and 1024 KiB of WRITE (scale 1)
    assert rec["fetch_scale"] == 2.0 and rec["write_scale"] == 1.0
    assert rec["hbm_bytes_per_launch"] == (1000 * 2 + 300) * 1024
    assert rec["commands"] == ["cmd"] and rec["workload"] == "w"
    assert len(rec["source_sha256"]) == 64


def test_launch_window(tmp_path):
    # five launches of one GEMM (written out of order) with durations 10, 20,
    # 30, 40, 50 us by start time; launches 1..3 average 30 us
    us = 1000
    write_trace(str(tmp_path), [
        (0, "void fs::gemm<0>(int)", 300 * us, 340 * us, 65536),
        (0, "void fs::gemm<0>(int)", 0, 10 * us, 65536),
        (0, "void fs::gemm<0>(int)", 100 * us, 120 * us, 65536),
        (0, "void fs::gemm<0>(int)", 400 * us, 450 * us, 65536),
        (0, "void fs::gemm<0>(int)", 200 * us, 230 * us, 65536),
        (0, "void fs::combine(int)", 500 * us, 505 * us, 4096),
    ])
    out = run(str(tmp_path), "--window", "gemm<0>", "1", "3")
    assert "gemm<0>: launches 1..3 (start order) average 30.00 us (min 20.00, max 40.00)" in out
    r = subprocess.run([sys.executable, TOOL, str(tmp_path), "--window", "gemm<0>", "3", "5"],
                       capture_output=True, text=True)
    assert r.returncode != 0 and "has 2 launches" in r.stderr


def test_split_launch_classes(tmp_path):
    # one kernel launched twice per step, a short pass (10 us) then a long
    # one (40 us), written out of order; --split tells them apart by launch
    # index modulo 2 in the trace, and in a counter run by dispatch order
    us = 1000
    rows = []
    for step in range(3):
        t = step * 1000 * us
        rows.append((0, "void fs::gemm<0>(int)", t + 500 * us, t + 540 * us, 65536))
        rows.append((0, "void fs::gemm<0>(int)", t, t + 10 * us, 65536))
    write_trace(str(tmp_path / "trace"), rows)
    out = run(str(tmp_path / "trace"), "--split", "gemm<0>", "2", "--window", "gemm<0> #1", "0", "3")
    assert "| gemm<0> #0 | 65536 | 3 | 10.00 | 10.00 | 10.00 |" in out
    assert "| gemm<0> #1 | 65536 | 3 | 40.00 | 40.00 | 40.00 |" in out
    assert "gemm<0> #1: launches 0..2 (start order) average 40.00 us" in out
    d = str(tmp_path / "fetch")
    os.makedirs(d)
    with open(os.path.join(d, "x_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Grid_Size", "Counter_Name",
                                          "Counter_Value"])
        w.writeheader()
        for i, kib in ((4, 700), (1, 100), (3, 100), (2, 700)):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": "void fs::gemm<0>(int)", "Grid_Size": 65536,
                        "Counter_Name": "FETCH_SIZE", "Counter_Value": kib})
    out = run(str(tmp_path / "trace"), "--split", "gemm<0>", "2", "--fetch", d)
    assert "| gemm<0> #0 | 65536 | 2 | 100 | - |" in out
    assert "| gemm<0> #1 | 65536 | 2 | 700 | - |" in out


def test_overlap_copy_stream(tmp_path):
    # long copies on both streams (the regular schedule's on the compute
    # stream 0, later in time): without --copy-stream the tool refuses;
    # with it, only stream 1's copy is reported and stream 0's is compute
    us = 1000
    write_trace(str(tmp_path), [
        (1, "paced_copy_kernel<uint4>", 0, 80 * us, 32768),
        (0, "void fs::gemm<0>(int)", 0, 60 * us, 65536),
        (0, "paced_copy_kernel<uint4>", 1000 * us, 1080 * us, 32768),
    ])
    r = subprocess.run([sys.executable, TOOL, str(tmp_path), "--overlap", "--copy-kernel", "paced_copy"],
                       capture_output=True, text=True)
    assert r.returncode != 0 and "several streams" in r.stderr
    out = run(str(tmp_path), "--overlap", "--copy-kernel", "paced_copy", "--copy-stream", "1")
    assert "copy stream 1: 1 copies" in out
    assert "| 1 | 80.0 | 75.0% | 75.0% | 75.0% | 20.0 |" in out
