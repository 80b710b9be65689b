"""Build the CPU oracle (plain C, gcc, OpenMP) into oracle/liboracle_nm.so.

Test infrastructure: compiled by the build entry point so that the checker is
available, never linked into the product library.
"""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "nm_oracle.c")
LIB_PATH = os.path.join(HERE, "liboracle_nm.so")


def build(out: str = LIB_PATH, src: str = SRC, extra=()) -> str:
    # -O3 without -ffast-math: the fp64 additions must keep their written
    # order (no reassociation), or the bit-exact brute-force pin would not hold.
    cmd = ["gcc", "-O3", "-std=c99", "-fPIC", "-shared", "-fopenmp",
           "-fno-fast-math", "-ffp-contract=off", *extra, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build())
