"""Compile the fp64 oracle (gc_oracle.c) into a shared library with gcc.

Test infrastructure: used by the test suite, the package build step and the
benchmark's CPU-baseline leg only.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "gc_oracle.c")
LIBRARY = os.path.join(HERE, "libgc_oracle.so")
# Plain IEEE arithmetic: no -ffast-math, no contraction into fused multiply-adds.
CFLAGS = ["-O2", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off", "-std=c11", "-Wall"]


def build_oracle(source: str = SOURCE, out: str = LIBRARY, extra=()) -> str:
    tmp = out + f".tmp{os.getpid()}"
    cmd = ["gcc", *CFLAGS, *extra, source, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build_oracle(*sys.argv[1:2]))
