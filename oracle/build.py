"""Build the oracle's C GEMM (TEST INFRASTRUCTURE ONLY) with gcc into oracle/liboracle_gemm.so.

-O3 with -ffp-contract=off and no fast-math: the compiler may vectorize across output
columns but keeps every dot product's fp64 sum in ascending k, unfused, so the results
are those of the plain loops. The ISA level stays x86-64-v2 rather than -march=native:
the library is built in one container and timed on another machine's host cores, and
instructions the build host has but the timing host lacks would stop it."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "ref_gemm.c")
LIB = os.path.join(HERE, "liboracle_gemm.so")


def build(force: bool = True) -> str:
    if not force and os.path.exists(LIB) and os.path.getmtime(LIB) >= os.path.getmtime(SRC):
        return LIB
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O3", "-march=x86-64-v2", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared", "-o", tmp, SRC]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(force="--force" in sys.argv or True))
