"""Host code and oracle under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only).  The kernels own disjoint columns by construction, so the device
side is covered by the bit-identity and padding tests; here the host side is:
the library's schedule generators, visit planner, its verifier (also on
corrupted plans) and the plan's scaling to byte offsets, skipped exchanges and LR schedule, and every round form of
the oracle in both precisions.  Both are built with the host compilers and
run as separate processes; any sanitizer report fails the test."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_11081_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, timeout):
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=timeout, env=ENV)
    assert r.returncode == 0, "%s failed:\n%s\n%s" % (cmd[0], r.stdout[-4000:], r.stderr[-4000:])
    return r


def test_host_code_under_sanitizers(tmp_path):
    cxx = shutil.which("g++")
    if not cxx:
        pytest.skip("no g++")
    exe = str(tmp_path / "sanitize_host")
    _run([cxx, "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(ROCM, "include"),
          "-I" + os.path.join(ROOT, "include"), "-I" + CSRC, os.path.join(ROOT, "tests", "sanitize_host.cpp"),
          os.path.join(CSRC, "plan.cpp"), os.path.join(CSRC, "topology.cpp"), os.path.join(CSRC, "schedule.cpp"),
          "-o", exe], 300)
    r = _run([exe], 600)
    assert "sanitize_host: ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr


@pytest.mark.parametrize("precision", ["f32", "f64"])
def test_oracle_under_sanitizers(tmp_path, precision):
    cc = shutil.which("gcc")
    if not cc:
        pytest.skip("no gcc")
    exe = str(tmp_path / ("sanitize_oracle_" + precision))
    defs = ["-DORACLE_FP64"] if precision == "f64" else []
    _run([cc, "-std=c11", *SAN, "-ffp-contract=off", *defs, os.path.join(ROOT, "tests", "sanitize_oracle.c"),
          os.path.join(ROOT, "oracle", "gasloc_oracle.c"), "-o", exe, "-lm"], 300)
    r = _run([exe], 600)
    assert "sanitize_oracle: ok" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
