"""bench.py end to end on the device, briefly (on the 25,557,032-element
workload, to keep it short): the one JSON line it prints keeps its contract
(metric, per-step throughput of the hard threshold, the roofline entry, the
Top-k and average rates, the oracle's CPU baselines, the workload)."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.timeout(300)
def test_bench_prints_one_contract_line():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "2",
                        "--steps", "3", "--warmup", "1", "--no-extra"],
                       capture_output=True, text=True, cwd=ROOT, timeout=280)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [x for x in r.stdout.splitlines() if x.strip()]
    assert len(lines) == 1
    b = json.loads(lines[0])
    assert b["metric"].startswith("G grad-elements/s")
    assert b["unit"] == "G grad-elements/s" and b["higher_is_better"] is True
    assert b["n_gpus"] == 1 and b["steps"] == 3 and b["warmup"] == 1
    assert b["value"] > 0 and b["ms_per_step"] > 0
    # value is d elements per hard-threshold step over the step time
    d = b["config"]["d"]
    assert d == 25_557_032
    assert b["value"] == pytest.approx(d / (b["ms_per_step"] * 1e-3) / 1e9, rel=2e-3)
    assert b["config"]["workload"].startswith("segments_25.6m: d=25,557,032")
    assert b["dtype"] == "f32" and b["data"] == "synthetic" and b["vs_baseline"] is None
    roof = b["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in roof
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"], abs=1e-3)
    assert 0.0 < roof["frac"] < 1.0
    assert roof["achieved"] == pytest.approx(
        roof["bytes_per_launch"] / (roof["launch_us"] * 1e-6) / 1e9, rel=2e-3)
    assert roof["launch_us"] == pytest.approx(b["ms_per_step"] * 1e3, rel=2e-3)
    for part in ("topk", "average"):
        assert 0.0 < b[part]["frac"] < 1.0 and b[part]["gbps"] > 0
    assert b["average"]["workers"] == 8 and b["average"]["status"] == 0
    for key, cores in (("cpu_baseline", None), ("cpu_baseline_1core", 1)):
        cpu = b[key]
        assert cpu["kind"] == "oracle" and cpu["value"] > 0 and cpu["cores"] >= 1
        assert cores is None or cpu["cores"] == cores
        assert cpu["unit"] == b["unit"] and cpu["sample"]
