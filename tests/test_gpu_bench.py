"""The benchmark's output on the GPU: a short run of bench.py (two timed
steps, no CPU leg, no extras) prints exactly one JSON line whose fields
follow the contract: the metric and its unit, one GPU, the steps asked for,
a value equal to d over the measured sparsify time, and the roofline object
of the dominant kernel."""
import json
import os
import subprocess
import sys

import pytest

from gpu_common import announce, need_gpu

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line():
    need_gpu()
    announce("bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-extras")
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "2",
                        "--warmup", "1", "--no-cpu-baseline", "--no-extras"],
                       capture_output=True, text=True, timeout=600)
    assert p.returncode == 0, p.stderr[-3000:]
    lines = [x for x in p.stdout.splitlines() if x.strip()]
    assert len(lines) == 1, p.stdout[-2000:]
    j = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in j, key
    assert j["n_gpus"] == 1 and j["steps"] == 2 and j["warmup"] == 1
    assert j["unit"] == "Gelem/s" and j["higher_is_better"] is True and j["dtype"] == "f32"
    assert j["data"] == "synthetic" and j["cpu_baseline"] is None and j["vs_baseline"] is None
    d = j["config"]["d"]
    assert d == 25_557_032 and "workload" in j["config"]
    assert j["value"] == pytest.approx(d / (j["sparsify_us"] * 1e3), rel=0.01)
    r = j["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert r["frac"] == pytest.approx(r["achieved"] / r["peak"], abs=1e-3)
    assert r["achieved"] == pytest.approx(
        r["algorithmic_bytes_per_launch"] / (r["mean_launch_us"] * 1e3), rel=0.01)
    assert 0.2 < r["frac"] < 1.0
