"""Host sanitizers: the CPU oracle (oracle/nm_oracle.c) and the library's host
half (packer, validator, size helpers in csrc/nmspmm_host.cpp) built from
source with AddressSanitizer and UndefinedBehaviorSanitizer (host code only,
plain gcc/g++: no GPU code is built here) and driven by
tests/sanitize/nm_sanitize_driver.cpp over ragged shapes, M up to 256, N = M,
dense and pruned inputs and the threaded packer.  Any out-of-bounds access,
leak or undefined behaviour fails the run."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


@pytest.mark.skipif(shutil.which("gcc") is None or shutil.which("g++") is None, reason="needs gcc and g++")
def test_oracle_and_host_packer_under_asan_ubsan(tmp_path):
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2503_01253_amd", "csrc"),
           "-I", "/opt/rocm/include", "-D__HIP_PLATFORM_AMD__"]
    objs = []
    # the oracle without OpenMP (its pragmas are then ignored: same results)
    o = str(tmp_path / "oracle.o")
    subprocess.run(["gcc", "-std=c99", *SAN, "-ffp-contract=off", "-c",
                    os.path.join(ROOT, "oracle", "nm_oracle.c"), "-o", o], check=True)
    objs.append(o)
    for name, src in (("host.o", os.path.join(ROOT, "paper_2503_01253_amd", "csrc", "nmspmm_host.cpp")),
                      ("driver.o", os.path.join(ROOT, "tests", "sanitize", "nm_sanitize_driver.cpp"))):
        o = str(tmp_path / name)
        subprocess.run(["g++", "-std=c++17", *SAN, *inc, "-c", src, "-o", o], check=True)
        objs.append(o)
    exe = str(tmp_path / "nm_sanitize")
    subprocess.run(["g++", *SAN, *objs, "-o", exe, "-pthread", "-lm"], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0 and "ALL OK" in r.stdout, r.stdout[-3000:] + r.stderr[-3000:]
