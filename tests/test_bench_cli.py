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
        "# HBM traffic\nFETCH_SIZE per launch (raw KiB): 120000.5\n"
        "WRITE_SIZE per launch (raw KiB): 200000.0\nscale (fetch, write): 2.0000, 1.0000\n"
        "hbm_bytes_per_launch: 451070927\nsource_digest: abc123\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    t = bench.read_traffic("update", "abc123")
    assert t == {"bytes": 451070927.0, "fetch_kib_raw": 120000.5, "write_kib_raw": 200000.0,
                 "fetch_scale": 2.0, "write_scale": 1.0}
    assert bench.read_traffic("update", "other") is None
    assert bench.read_traffic("stream", "abc123") is None


def test_source_digest_is_stable():
    a = bench.kernel_source_digest()
    assert a == bench.kernel_source_digest() and len(a) == 16


def test_profile_summaries(tmp_path, capsys):
    """The --summarize-stats / --summarize-pmc readers of rocprofv3 CSV output
    (the commands the profile summaries quote)."""
    stats = tmp_path / "s.csv"
    stats.write_text('"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs"\n'
                     '"tkef::k_stream(tkef::TileDesc const*, int)",25,1325000,53000,13.0,51000,56000\n'
                     '"void at::native::foo(int)",3,300,100,0.1,90,110\n')
    assert bench.summarize_stats(str(stats)) == 0
    out = capsys.readouterr().out
    assert "tkef::k_stream" in out and "53.00" in out and "at::native" not in out
    pmc = tmp_path / "p.csv"
    rows = ['"Dispatch_Id","Kernel_Name","Counter_Name","Counter_Value"']
    for dsp, v in ((1, 10.0), (1, 5.0), (2, 30.0)):
        rows.append(f'"{dsp}","void tkef::k_seg<false>(tkef::ListsArg)","FETCH_SIZE","{v}"')
    rows.append('"3","void tkef::k_seg<false>(tkef::ListsArg)","WRITE_SIZE","99"')
    pmc.write_text("\n".join(rows) + "\n")
    assert bench.summarize_pmc(str(pmc), "FETCH_SIZE") == 0
    out = capsys.readouterr().out
    assert "tkef::k_seg<false>" in out and " 2 " in out and "22.5" in out


def test_host_description():
    assert bench.usable_cores() >= 1
    assert isinstance(bench.cpu_model(), str) and bench.cpu_model()
