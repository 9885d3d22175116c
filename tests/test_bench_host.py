"""Host-side logic of bench.py: the rocprofv3 summary parsers and the
one-GPU guard (no GPU needed)."""
import csv
import argparse
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

HT = "void efs::ht_fused_kernel<true, false>(float const*, float*, long, float)"
HT_STATS = "void efs::ht_fused_kernel<true, true>(float const*, float*, long, float)"
COPY = "efs::(anonymous namespace)::copy_kernel(float const*, float*, long, unsigned int)"
OTHER = "efs::(anonymous namespace)::topk_step3_kernel(float*, long)"


def _write_csv(path, fields, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=fields)
        w.writeheader()
        for r in rows:
            w.writerow(r)


def _trace(folder, dispatches):
    """dispatches: (kernel name, duration in ns), in launch order."""
    t, rows, by = 1000, [], {}
    for name, dur in dispatches:
        rows.append({"Kernel_Name": name, "Start_Timestamp": t, "End_Timestamp": t + dur})
        t += dur + 500
        by.setdefault(name, []).append(dur)
    _write_csv(os.path.join(folder, "run_kernel_trace.csv"),
               ["Kernel_Name", "Start_Timestamp", "End_Timestamp"], rows)
    stats = [{"Name": n, "Calls": len(v), "TotalDurationNs": sum(v), "AverageNs": sum(v) / len(v),
              "MinNs": min(v), "MaxNs": max(v)} for n, v in by.items()]
    _write_csv(os.path.join(folder, "run_kernel_stats.csv"),
               ["Name", "Calls", "TotalDurationNs", "AverageNs", "MinNs", "MaxNs"], stats)


def test_parse_trace_finds_the_timed_run(tmp_path):
    # hard-threshold launches interleaved with others, the telemetry variant
    # back to back, then the 4 plain launches of the timed steps back to back
    seq = []
    for _ in range(3):
        seq += [(HT, 70_000), (OTHER, 9_000)]
    seq += [(HT_STATS, 60_000)] * 4
    seq += [(OTHER, 9_000)]
    seq += [(HT, 50_000), (HT, 52_000), (HT, 48_000), (HT, 50_000)]
    seq += [(OTHER, 9_000), (HT, 90_000)]
    _trace(str(tmp_path), seq)
    out = bench.parse_trace(str(tmp_path), 4)
    line = [x for x in out.splitlines() if "timed steps" in x]
    assert len(line) == 1
    assert "avg 50.00 us, min 48.00, max 52.00" in line[0]
    # the whole-run table averages every dispatch of the kernel
    row = [x for x in out.splitlines() if x.startswith("ht_fused_kernel<true, false>")][0]
    assert float(row.split()[3]) == pytest.approx((3 * 70 + 200 + 90) / 8.0)


def test_parse_trace_says_when_no_run_matches(tmp_path):
    _trace(str(tmp_path), [(HT, 50_000), (OTHER, 9_000), (HT, 50_000)])
    assert "no run of 20 back-to-back" in bench.parse_trace(str(tmp_path), 20)


def _pmc(folder, counter, values):
    # rows written out of dispatch order: the parser sorts them
    os.makedirs(folder)
    rows = [{"Dispatch_Id": i + 1, "Kernel_Name": n, "Counter_Name": counter, "Counter_Value": v}
            for i, (n, v) in enumerate(values)]
    _write_csv(os.path.join(folder, "run_counter_collection.csv"),
               ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"], rows[::-1])


def test_parse_pmc_scales_by_the_copy_probe(tmp_path):
    d = 1 << 20
    # the copy probe moves 4d bytes each way; its counters read 2x (fetch)
    # and 1x (write) of that, so the kernel's readings are scaled by 1/2, 1
    fetch, write = str(tmp_path / "f"), str(tmp_path / "w")
    # two hard-threshold launches on the workload, then a later small one
    # (the average's payloads) that the per-launch figure leaves out
    _pmc(fetch, "FETCH_SIZE", [(HT, 16384.0), (HT, 16384.0), (COPY, 8192.0), (HT, 8.0)])
    _pmc(write, "WRITE_SIZE", [(HT, 4096.0), (HT, 4096.0), (COPY, 4096.0), (OTHER, 1.0),
                               (HT, 4.0)])
    res = bench.parse_pmc(fetch, write, d, 2)
    assert res["FETCH_SIZE"]["scale"] == pytest.approx(0.5)
    assert res["WRITE_SIZE"]["scale"] == pytest.approx(1.0)
    assert res["ht_bytes_per_launch"] == pytest.approx(16384 * 1024 * 0.5 + 4096 * 1024)
    text = bench.format_traffic(res, "a workload", argparse.Namespace(warmup=0, steps=1))
    assert "ht_bytes_per_launch %d" % round(res["ht_bytes_per_launch"]) in text
    # the other kernels get the same scales: topk_step3 fetched nothing, wrote 1 KiB
    step3 = [x for x in text.splitlines() if "topk_step3_kernel" in x]
    assert len(step3) == 1 and "0.00 +      0.00 MB  (1)" in step3[0]
    ht_line = [x for x in text.splitlines()
               if x.startswith("#   ht_fused_kernel<true, false>")][0]
    every = ((2 * 16384 + 8) / 3 * 1024 * 0.5 / 1e6, (2 * 4096 + 4) / 3 * 1024 / 1e6)
    assert "%9.2f + %9.2f MB" % every in ht_line
    assert "kernel_source_sha256 " + bench.kernel_source_digest() in text


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_parse_trace_last_takes_each_kernels_last_dispatches(tmp_path):
    # warm-up calls slower than the timed ones: only each kernel's last n
    # dispatches count, and kernels are ordered by their average
    P1 = "void efs::(anonymous namespace)::seg_pass1_kernel<true>(float const*, float*)"
    FIN = "void efs::(anonymous namespace)::seg_final_kernel<3840>(float*, int*)"
    seq = []
    for _ in range(5):
        seq += [(P1, 900_000), (FIN, 400_000)]
    for d in (100_000, 120_000, 110_000):
        seq += [(P1, d), (FIN, 40_000)]
    _trace(str(tmp_path), seq)
    out = bench.parse_trace_last(str(tmp_path), 3).splitlines()
    assert out[1].split() == ["seg_pass1_kernel<true>", "3", "110.00", "100.00", "120.00"]
    assert out[2].split() == ["seg_final_kernel<3840>", "3", "40.00", "40.00", "40.00"]
