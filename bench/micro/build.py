"""Build the roof micro-benchmarks (bench/micro/nm_micro.hip) into
bench/micro/libnm_micro.so for gfx950, in-tree.

    python bench/micro/build.py
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "nm_micro.hip")
LIB_PATH = os.path.join(HERE, "libnm_micro.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build(out: str = LIB_PATH, verbose: bool = False) -> str:
    # the same device flags as the product library (packed fp32 VALU off)
    cmd = [HIPCC, "-O3", "-std=c++17", "-fPIC", "-shared", "-fvisibility=hidden", "--offload-arch=gfx950",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), SRC, "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
