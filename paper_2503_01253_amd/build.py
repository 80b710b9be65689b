"""Build libnmspmm.so (HIP kernels + C ABI) for gfx950, in-tree, and its
debug twin libnmspmm_poison.so (the same sources with NMSPMM_POISON_LDS=1:
every LDS fill is preceded by NaN in its destination, so that a missing wait
or barrier shows up as a wrong result in the tests that load it).

    python -m paper_2503_01253_amd.build
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_PATH = os.path.join(PKG, "libnmspmm.so")
POISON_LIB_PATH = os.path.join(PKG, "libnmspmm_poison.so")
SOURCES = sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + [os.path.join(CSRC, "nmspmm_host.cpp")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed fp32 VALU ops (v_pk_*_f32) are switched off for every device
# compilation: the fp32 math of these kernels runs on MFMA and scalar VALU.
DEVICE_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-Wall", "-Wno-unused-result"]


def _compile(src: str, verbose: bool, defines=(), tag: str = "") -> str:
    obj = os.path.join(CSRC, os.path.basename(src) + tag + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [HIPCC, *COMMON_FLAGS, *DEVICE_FLAGS, *defines, "-I", INCLUDE, "-I", CSRC, *lang, "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True)
    return obj


def build(out: str = LIB_PATH, verbose: bool = False, jobs: int = 0, defines=(), tag: str = "") -> str:
    """Compile every source (in parallel) and link the shared library."""
    jobs = jobs or min(len(SOURCES), os.cpu_count() or 1, 16)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, defines, tag), SOURCES))
    link = [HIPCC, *DEVICE_FLAGS, "-shared", "-fPIC", *objs, "-o", out + ".tmp"]
    if verbose:
        print(" ".join(link), file=sys.stderr)
    subprocess.run(link, check=True)
    os.replace(out + ".tmp", out)
    for obj in objs:
        os.remove(obj)
    return out


def build_poison(verbose: bool = False, jobs: int = 0) -> str:
    """The debug twin with NaN-poisoned LDS fills (tests only)."""
    return build(POISON_LIB_PATH, verbose, jobs, defines=("-DNMSPMM_POISON_LDS=1",), tag=".poison")


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_poison())
