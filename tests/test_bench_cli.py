"""Host-side checks of bench.py: the one-GPU contract and the rule that the
counter-based traffic figure is reported only for the kernel sources it was
measured on."""
from __future__ import annotations

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr
    assert p.stdout == ""


def test_traffic_needs_matching_source_digest(tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "traffic_update_resnet50.txt").write_text(
        "# HBM traffic\nhbm_bytes_per_launch: 451070927\nsource_digest: abc123\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.read_traffic("update", "abc123") == 451070927.0
    assert bench.read_traffic("update", "other") is None
    assert bench.read_traffic("stream", "abc123") is None


def test_source_digest_is_stable():
    a = bench.kernel_source_digest()
    assert a == bench.kernel_source_digest() and len(a) == 16
