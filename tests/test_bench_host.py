"""Host-side parts of bench.py that need no GPU: the one-GPU guard and the
HBM-traffic summary built from rocprofv3 counter files."""

import csv
import json
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def _counter_csv(path, counter, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                          "Counter_Value"])
        w.writeheader()
        for i, (name, value) in enumerate(rows):
            w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter,
                        "Counter_Value": value})


def test_traffic_summary_counts_only_the_step_dispatches(tmp_path):
    kmv = "void ep::(anonymous namespace)::kmv_kernel<0, 4, true, 1, 32, false, 8>(ep::KmvArgs)"
    sub = "void ep::(anonymous namespace)::kmv_subsample_kernel<0, 4, true, 1, 32, false, 8>"
    copy = "__amd_rocclr_copyBuffer"
    # three step launches, then two prediction launches of the same kernel
    # on another shape; the 1 GiB calibration copies read as 0.5 GiB
    fetch = [(kmv, 1000.0), (sub, 7.0), (kmv, 1000.0), (sub, 7.0), (kmv, 1000.0), (sub, 7.0),
             (kmv, 5000.0), (kmv, 5000.0), (copy, 524288.0), (copy, 524288.0), (copy, 8.0)]
    write = [(kmv, 10.0), (sub, 1.0), (kmv, 10.0), (sub, 1.0), (kmv, 10.0), (sub, 1.0),
             (kmv, 50.0), (kmv, 50.0), (copy, 1048576.0), (copy, 1048576.0), (copy, 8.0)]
    fcsv, wcsv, out = tmp_path / "f.csv", tmp_path / "w.csv", tmp_path / "t.json"
    _counter_csv(fcsv, "FETCH_SIZE", fetch)
    _counter_csv(wcsv, "WRITE_SIZE", write)
    text = bench.traffic_summary(str(fcsv), str(wcsv), "w", "kmv_kernel", 3, "note",
                                 out_path=str(out))
    rec = json.loads(out.read_text())["w | kmv_kernel"]
    assert rec["read_factor"] == 2.0 and rec["write_factor"] == 1.0
    assert rec["fetch_kib"] == 1000.0 and rec["write_kib"] == 10.0
    assert rec["bytes_per_launch"] == (1000.0 * 2 + 10.0) * 1024
    assert rec["source_sha"] == bench.kernel_source_sha("kmv_kernel")
    assert "its first 3 dispatches" in text


def test_code_hash_ignores_comments_only():
    src = "int f(int a) { // one\n  return a + 1; /* two\n lines */ }\n"
    same = "int f(int a) {\n  // other words\n  return a + 1;\n}"
    changed = "int f(int a) { return a + 2; }"
    assert bench.code_text(src) == bench.code_text(same)
    assert bench.code_text(src) != bench.code_text(changed)
    assert "//" not in bench.code_text(src) and "/*" not in bench.code_text(src)
