"""The gfx950 code objects of the library as built here (no GPU): every HIP
source has its device binary, and none of them holds packed-fp32 arithmetic
(the device pass disables that target feature; the host pass is not given
it)."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2606_11081_amd import build as lib_build

ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
BUNDLER = os.path.join(ROCM, "llvm", "bin", "clang-offload-bundler")
OBJDUMP = os.path.join(ROCM, "llvm", "bin", "llvm-objdump")
PACKED_FP32 = re.compile(r"\bv_pk_(add|mul|fma)_f32\b")


def _disassemble(src, tmp_path):
    fatbin = lib_build.device_binary(src)
    if not os.path.exists(fatbin):
        pytest.skip("library not built")
    co = str(tmp_path / (os.path.splitext(src)[0] + ".co"))
    subprocess.run([BUNDLER, "--unbundle", "--type=o", "--targets=hipv4-amdgcn-amd-amdhsa--gfx950",
                    "--input=" + fatbin, "--output=" + co], check=True, capture_output=True)
    return subprocess.run([OBJDUMP, "-d", co], check=True, capture_output=True, text=True).stdout


@pytest.mark.skipif(not (os.path.exists(BUNDLER) and os.path.exists(OBJDUMP)), reason="ROCm LLVM tools absent")
@pytest.mark.parametrize("src", [s for s in lib_build.SOURCES if s.endswith(".hip")])
def test_device_code_has_no_packed_fp32_arithmetic(src, tmp_path):
    text = _disassemble(src, tmp_path)
    assert "s_endpgm" in text  # it is the kernels' code
    found = sorted(set(m.group(0) for m in PACKED_FP32.finditer(text)))
    assert not found, (src, found)


def test_host_objects_embed_the_device_binaries():
    assert shutil.which("hipcc") or os.path.exists(os.path.join(ROCM, "bin", "hipcc"))
    for src in lib_build.SOURCES:
        if src.endswith(".hip") and os.path.exists(lib_build.device_binary(src)):
            obj = os.path.join(lib_build.BUILD, os.path.splitext(src)[0] + ".o")
            data = open(obj, "rb").read()
            assert b"__CLANG_OFFLOAD_BUNDLE__" in data, src
