"""Host logic of the benchmark (CPU only): the rocprofv3 summaries it writes under
profiles/ (kernel table, copy-calibrated HBM bytes per dispatch, the attention traffic
record and its staleness check), and its refusal of more than one GPU.

The summaries are built from small synthetic CSV files laid out as rocprofv3 writes
them, in a temporary directory; bench.ROOT is pointed there, so no committed profile
is touched.
"""
import csv
import json
import os
import subprocess
import sys

import pytest

import bench

ATTN = "void tu::(anonymous namespace)::k_attn<256>(tu::AttnArgs, tu::AttnOrder)"
PART = "void tu::(anonymous namespace)::k_probe_part<256>(tu::ProbeArgs)"


def _write_csv(path, fields, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=fields)
        w.writeheader()
        for r in rows:
            w.writerow(r)


def _rocprof_dir(root, fetch_kib, write_kib, calib_fetch_kib, calib_write_kib):
    """trace/, calib_*/ and pmc_*/ outputs: two kernels, two dispatches each."""
    out = os.path.join(root, "prof")
    _write_csv(os.path.join(out, "trace", "run_kernel_stats.csv"),
               ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs"],
               [{"Name": ATTN, "Calls": 2, "TotalDurationNs": 4000, "AverageNs": 2000, "Percentage": 80,
                 "MinNs": 1900, "MaxNs": 2100},
                {"Name": PART, "Calls": 2, "TotalDurationNs": 1000, "AverageNs": 500, "Percentage": 20,
                 "MinNs": 450, "MaxNs": 550},
                {"Name": "some_torch_kernel", "Calls": 1, "TotalDurationNs": 10, "AverageNs": 10,
                 "Percentage": 0, "MinNs": 10, "MaxNs": 10}])
    for kind, per, calib in (("FETCH_SIZE", fetch_kib, calib_fetch_kib), ("WRITE_SIZE", write_kib, calib_write_kib)):
        rows = []
        for name, kib in per.items():
            for d in range(2):   # median over the dispatches
                rows.append({"Kernel_Name": name, "Counter_Value": kib + (d - 0.5) * 2})
        _write_csv(os.path.join(out, f"pmc_{kind}", "run_counter_collection.csv"), ["Kernel_Name", "Counter_Value"],
                   rows)
        _write_csv(os.path.join(out, f"calib_{kind}", "run_counter_collection.csv"),
                   ["Kernel_Name", "Counter_Value"],
                   [{"Kernel_Name": "copy", "Counter_Value": calib}, {"Kernel_Name": "fill", "Counter_Value": 12.0}])
    return out


@pytest.fixture()
def fake_root(tmp_path, monkeypatch):
    root = tmp_path / "repo"
    (root / "profiles").mkdir(parents=True)
    # the traffic record hashes the attention kernel's sources: copy them in
    for src in bench.KERNEL_SOURCES["attention"]:
        dst = root / src
        dst.parent.mkdir(parents=True, exist_ok=True)
        dst.write_bytes(open(os.path.join(bench.ROOT, src), "rb").read())
    monkeypatch.setattr(bench, "ROOT", str(root))
    return root


def test_update_profile_summary_and_traffic_record(fake_root):
    # FETCH_SIZE counts half the bytes read (calibration 131,072 KiB for a 256 MiB copy)
    out = _rocprof_dir(str(fake_root), {ATTN: 1024.0, PART: 256.0}, {ATTN: 512.0}, 131072.0, 262144.0)
    bench.summarize_profile(out, 4)
    md = (fake_root / "profiles" / "update_stack_config4.md").read_text()
    assert "| k_attn<256> | 2 | 2.00 | 1.90 | 2.10 |" in md
    assert "some_torch_kernel" not in md
    assert "| k_attn<256> | 2.00 | 0.50 |" in md       # 1024 KiB x 2 read, 512 KiB written
    rec = json.loads((fake_root / "profiles" / "traffic_config4.json").read_text())
    assert rec["fetch_bytes_per_launch"] == 2 * 1024 * 1024 and rec["write_bytes_per_launch"] == 512 * 1024
    wl = rec["workload"]
    t = bench.measured_traffic("attention", 4, wl)
    assert t is not None and t["bytes_per_launch"] == 2 * 1024 * 1024 + 512 * 1024
    # another workload, or a source changed since the counters were taken: no traffic
    assert bench.measured_traffic("attention", 4, wl + " (other)") is None
    src = fake_root / bench.KERNEL_SOURCES["attention"][0]
    src.write_bytes(src.read_bytes() + b"\n// changed\n")
    assert bench.measured_traffic("attention", 4, wl) is None


def test_diagnostics_profile_summary(fake_root):
    out = _rocprof_dir(str(fake_root), {PART: 32768.0}, {PART: 4096.0}, 131072.0, 262144.0)
    row = {"config": "config 4: x", "attention_diagnostics": {"live_rows": 65536, "probe_ms": 0.6}}
    with open(os.path.join(out, "plain.log"), "w") as f:
        f.write("[bench] building\n" + json.dumps(row) + "\n")
    bench.summarize_diagnostics(out, 4)
    md = (fake_root / "profiles" / "attention_diagnostics_config4.md").read_text()
    assert "| k_probe_part<256> | 2 | 0.50 | 0.45 | 0.55 |" in md
    assert "| k_probe_part<256> | 64.00 | 4.00 |" in md  # 32,768 KiB counted = 64 MiB read
    assert "64.0 MiB (65,536 live rows" in md
    assert '"probe_ms": 0.6' in md
    assert "--only-diagnostics" in md and "--summarize-diagnostics" in md


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(bench.ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]
