"""The C ABI from plain C (no GPU): include/gasloc.h and gasloc_probe.h compile as C99 with
warnings as errors, a C program links against libgasloc.so and its host-side
calls agree with the oracle."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2606_11081_amd")


def test_plain_c_consumer(tmp_path):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    if not os.path.exists(os.path.join(LIBDIR, "libgasloc.so")):
        pytest.skip("libgasloc.so not built")
    exe = str(tmp_path / "c_consumer")
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I" + os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c_consumer.c"), "-L" + LIBDIR, "-lgasloc",
                    "-Wl,-rpath," + LIBDIR, "-lm", "-o", exe], check=True, capture_output=True)
    out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout.splitlines()
    lines = dict(line.split("=", 1) if "=" in line.split()[0] else (line.split()[0], line) for line in out)

    rp, col, val = oracle.topology_csr("exponential", 8, 3, 0)
    row0 = " ".join("%d:%g" % (c, v) for c, v in zip(col[rp[0]:rp[1]], val[rp[0]:rp[1]]))
    assert out[0] == "exponential n=8 nnz=%d row0= %s" % (len(col), row0)
    assert lines["validate"] == "0"       # GASLOC_OK
    assert lines["validate_bad"] == "1"   # GASLOC_EINVAL: a row that does not sum to 1
    alive = np.array([i != 5 for i in range(8)], np.uint8)
    srp, scol, sval = oracle.skip_exchanges((rp, col, val), 8, alive)
    row5 = " ".join("%d:%g" % (c, v) for c, v in zip(scol[srp[5]:srp[6]], sval[srp[5]:srp[6]]))
    assert out[3] == "dead5 row5= " + row5
    lr = [float(v) for v in lines["lr"].split()]
    f = lambda v: float(np.float32(v))  # the C program passes float arguments
    expect = [oracle.lr_schedule(f(1e-3), s, 100, f(0.1), f(0.01), 0.0) for s in (0, 10, 99)]
    assert [np.float32(v) for v in lr] == [np.float32(v) for v in expect]
    assert lines["probe_mix"] == "1"    # GASLOC_EINVAL: unsupported mix of streams
    assert lines["probe_count"] == "1"  # GASLOC_EINVAL: count outside [1, 2^31)
    assert lines["probe_threads"] == "1"  # GASLOC_EINVAL: threads not 64, 128 or 256


@pytest.mark.gpu
def test_c_program_runs_rounds_on_the_gpu(tmp_path):
    # whole rounds through the C ABI from a C program (hipMalloc'd buffers, no
    # Python or torch in that process), bit-identical to the fp32 oracle
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    exe = str(tmp_path / "c_device_consumer")
    subprocess.run([cc, "-std=c11", "-Wall", "-Wextra", "-Werror", "-O2", "-ffp-contract=off", "-D__HIP_PLATFORM_AMD__",
                    "-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(rocm, "include"),
                    os.path.join(ROOT, "tests", "c_device_consumer.c"), os.path.join(ROOT, "oracle", "gasloc_oracle.c"),
                    "-L" + LIBDIR, "-lgasloc", "-Wl,-rpath," + LIBDIR, "-L" + os.path.join(rocm, "lib"), "-lamdhip64",
                    "-Wl,-rpath," + os.path.join(rocm, "lib"), "-lm", "-o", exe], check=True, capture_output=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c_device_consumer: ok" in r.stdout
