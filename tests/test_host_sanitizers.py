"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The C oracle, built with gcc -fsanitize=address,undefined, run over small
  seeded cases by tests/sanitize/oracle_driver.c (selection against the rank
  definition at every k, signed zeros, infinities, subnormals, NaN
  rejection, dyadic aggregate and update identities, error paths).
* The library's host code (argument checks, plan and workspace layout,
  descriptor tables, the one-shot calls' error paths), built with the
  sanitizers on the host side only (each -fsanitize= behind -Xarch_host: the
  GPU code is neither instrumented nor launched) and driven through the C
  ABI by tests/sanitize/host_abi_driver.cpp on this machine without a GPU,
  where calls that pass every check end in the HIP runtime's no-device error.

Any sanitizer report aborts the driver (-fno-sanitize-recover=all); the
drivers' exit status counts their failed checks.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = "/opt/rocm/bin/hipcc"


def _run(exe, leaks):
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = f"detect_leaks={1 if leaks else 0}:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1"
    p = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    out = p.stdout + p.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert p.returncode == 0, out[-4000:]
    return out


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", "-ffp-contract=off",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-fno-omit-frame-pointer",
                    os.path.join(ROOT, "oracle", "tkef_oracle.c"),
                    os.path.join(SAN, "oracle_driver.c"), "-lm", "-o", exe],
                   check=True, capture_output=True, timeout=300)
    assert "0 failed checks" in _run(exe, leaks=True)


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_host_abi_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "host_abi_driver")
    csrc = os.path.join(ROOT, "paper_2010_10458_amd", "csrc")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           "-I" + os.path.join(ROOT, "include"), "-I" + csrc,
           os.path.join(csrc, "tkef_kernels.hip"), os.path.join(csrc, "tkef_api.cpp"),
           os.path.join(SAN, "host_abi_driver.cpp"), "-o", exe]
    p = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert p.returncode == 0, p.stderr[-4000:]
    # (leak checking off: the HIP runtime that the calls reaching it
    # initialise is not this library's code)
    assert "0 failed checks" in _run(exe, leaks=False)
