"""Compile the C oracle into ``oracle/liboracle.so`` with gcc (OpenMP, fp64, no fast-math).

Test infrastructure only.  ``build(src, out)`` is also used by the tests to
compile deliberately broken copies of the oracle into a temporary folder.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "kmeans_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

# -O2 without -ffast-math or -ffp-contract=fast: every fp64 operation is rounded
# as written, in the order written.
CFLAGS = ["-O2", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-std=c11", "-Wall"]


def build(src: str = SRC, out: str = LIB) -> str:
    tmp = out + f".tmp{os.getpid()}"
    cmd = ["gcc", *CFLAGS, src, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(*(sys.argv[1:3])))
