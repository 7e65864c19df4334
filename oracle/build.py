"""Build the plain-C oracle into two shared objects (test infrastructure).

liboracle_f32.so : fp32 arithmetic (the workloads' parameter/state precision),
                   bf16 parameter storage supported.
liboracle_f64.so : fp64 arithmetic and fp64 state.

Both are compiled with -O2 and -ffp-contract=off, no intrinsics, no OpenMP.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "gasloc_oracle.c")
LIBS = {
    "f32": os.path.join(HERE, "liboracle_f32.so"),
    "f64": os.path.join(HERE, "liboracle_f64.so"),
}


def build(verbose=False):
    base = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
            "-Wall", "-Wextra"]
    for tag, out in LIBS.items():
        cmd = list(base)
        if tag == "f64":
            cmd.append("-DORACLE_FP64")
        cmd += [SRC, "-o", out + ".tmp", "-lm"]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(out + ".tmp", out)
    return dict(LIBS)


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
