"""Compile libgasloc.so (HIP kernels for gfx950 + host runtime) in-tree.

Every HIP translation unit is built with -ffp-contract=off (no fused
multiply-add: the op order of the round is part of its definition).  A .hip
file is compiled in two passes: the device pass for gfx950 with packed-fp32
instructions disabled (a gfx950 target feature), then the host pass, which
embeds the device binary and is not given that feature (the host target does
not know it).
"""
import hashlib
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libgasloc.so")
SOURCES = ["adamw.hip", "round_phase.hip", "round_planned.hip", "round_shared.hip", "reductions.hip",
           "stream_probe.hip", "runtime.cpp", "topology.cpp", "schedule.cpp", "plan.cpp"]
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-ffp-contract=off",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC]
HIP = ["-x", "hip", "--offload-arch=" + ARCH, "-fno-gpu-rdc"]
DEVICE_ONLY = ["--cuda-device-only", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HOST_CXX = [os.path.join(ROCM, "llvm", "bin", "clang++"), "-D__HIP_PLATFORM_AMD__",
            "-I", os.path.join(ROCM, "include")]


def sources_sha():
    """SHA-256 (first 16 hex digits) of every source the library is compiled
    from: csrc/ and include/, files in name order, each name then its bytes."""
    h = hashlib.sha256()
    for d in (CSRC, os.path.join(ROOT, "include")):
        for name in sorted(os.listdir(d)):
            if name.endswith((".hip", ".cpp", ".h")):
                h.update(name.encode())
                with open(os.path.join(d, name), "rb") as f:
                    h.update(f.read())
    return h.hexdigest()[:16]


def build_info():
    """What gasloc_build_info() of a library built now returns."""
    return "sources %s; %s; -O3 -ffp-contract=off; device pass without packed-fp32" % (sources_sha(), ARCH)


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def device_binary(src):
    """The bundled gfx950 code object of a .hip source (written by build())."""
    return os.path.join(BUILD, os.path.splitext(src)[0] + ".hipfb")


def _compile(src, verbose, info):
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    path = os.path.join(CSRC, src)
    if src == "runtime.cpp":
        return _run(HOST_CXX + COMMON + ['-DGASLOC_BUILD_INFO="%s"' % info, "-c", path, "-o", obj], verbose) or obj
    if src.endswith(".hip"):
        fatbin = device_binary(src)
        _run(["hipcc"] + COMMON + HIP + DEVICE_ONLY + ["-c", path, "-o", fatbin], verbose)
        _run(["hipcc"] + COMMON + HIP + ["--cuda-host-only", "-Xclang", "-fcuda-include-gpubinary", "-Xclang",
                                         fatbin, "-c", path, "-o", obj], verbose)
    else:  # host-only C++ against the HIP runtime API
        _run(HOST_CXX + COMMON + ["-c", path, "-o", obj], verbose)
    return obj


def build(verbose=False):
    os.makedirs(BUILD, exist_ok=True)
    info = build_info()
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, info), SOURCES))
    tmp = LIB + ".tmp"
    _run(["hipcc", "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs, verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
