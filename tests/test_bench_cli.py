"""Host-side logic of bench.py: the one-GPU refusal and the rocprofv3 summaries
that the bench line's roofline figures come from (no GPU involved)."""
import csv
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=300)


def _write_counters(path, counter, rows):
    with open(path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value", "Grid_Size"])
        wr.writeheader()
        for name, kib in rows:
            wr.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": kib, "Grid_Size": 256})


def test_more_than_one_gpu_is_refused():
    r = _bench("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_trace_summary_means(tmp_path):
    p = tmp_path / "trace.csv"
    with open(p, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        wr.writeheader()
        for s, e in ((1000, 31000), (50000, 80000)):                    # 30 us twice
            wr.writerow({"Kernel_Name": "decode_stream_kernel", "Start_Timestamp": s, "End_Timestamp": e})
        wr.writerow({"Kernel_Name": "decode_merge_kernel", "Start_Timestamp": 0, "End_Timestamp": 4000})
    r = _bench("--summarize-trace", str(p))
    assert r.returncode == 0, r.stderr
    line = next(ln for ln in r.stdout.splitlines() if ln.endswith("decode_stream_kernel"))
    calls, mean, lo, hi, total = line.split()[:5]
    assert (int(calls), float(mean), float(lo), float(hi), float(total)) == (2, 30.0, 30.0, 30.0, 0.06)


def test_pmc_summary_scales_by_the_calibration_copy(tmp_path):
    # The calibration copy of 1 MiB reads 512 KiB and writes 1024 KiB by the counters: the
    # fetch scale is 2 and the write scale 1.  Per layer the split-K kernel fetches 1000 KiB
    # and writes 5 KiB (counter units), so its launch moves (1000 * 2 + 5) * 1024 bytes; the
    # combine kernel's 10 KiB are recorded apart.
    f, w, out = tmp_path / "f.csv", tmp_path / "w.csv", tmp_path / "traffic.json"
    _write_counters(f, "FETCH_SIZE", [("__amd_rocclr_copyBuffer", 512.0), ("decode_stream_kernel", 1000.0),
                                      ("decode_stream_kernel", 1000.0), ("decode_merge_kernel", 10.0)])
    _write_counters(w, "WRITE_SIZE", [("__amd_rocclr_copyBuffer", 1024.0), ("decode_stream_kernel", 5.0),
                                      ("decode_stream_kernel", 5.0), ("decode_merge_kernel", 0.0)])
    r = _bench("--summarize-pmc", str(f), str(w), "--calibrate-copy-mib", "1", "--traffic-json", str(out))
    assert r.returncode == 0, r.stderr
    rec = json.loads(out.read_text())
    assert rec["fetch_scale"] == 2.0 and rec["write_scale"] == 1.0
    assert rec["bytes_per_launch"] == (1000 * 2 + 5) * 1024
    assert rec["combine_bytes"] == 10 * 2 * 1024
    assert rec["kernels"] == ["decode_stream_kernel"]
