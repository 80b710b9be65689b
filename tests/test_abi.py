"""CPU tests of the C ABI: the library loads, exports every declared symbol,
packs exactly like the oracle, validates patterns and rejects bad arguments
before touching the GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2503_01253_amd as nm
from nm_workloads import make_inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "nmspmm.h")).read()
    return sorted(set(re.findall(r"NMSPMM_API\s+[\w\s\*]*?\b(nmspmm_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_symbols()
    assert len(names) == 17
    assert sorted(nm.EXPORTS) == names
    L = nm.lib()
    for name in names:
        assert hasattr(L, name), name
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value


def test_micro_library_exports_every_declared_symbol():
    """The roof micro-benchmarks' library (bench/micro) exports what
    include/nm_micro.h declares."""
    text = open(os.path.join(ROOT, "include", "nm_micro.h")).read()
    names = sorted(set(re.findall(r"NM_MICRO_API\s+[\w\s\*]*?\b(nm_micro_\w+)\s*\(", text)))
    assert names == ["nm_micro_hbm_read", "nm_micro_mfma_f32", "nm_micro_mfma_f32_flops"]
    L = ctypes.CDLL(os.path.join(ROOT, "bench", "micro", "libnm_micro.so"))
    for name in names:
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value, name
    L.nm_micro_mfma_f32_flops.argtypes = [ctypes.c_int, ctypes.c_int]
    L.nm_micro_mfma_f32_flops.restype = ctypes.c_double
    assert L.nm_micro_mfma_f32_flops(10, 3) == 2 * 32 * 32 * 2 * 8 * 10 * 4 * 3
    L.nm_micro_hbm_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    assert L.nm_micro_hbm_read(0x1000, 100, 0x1000, 8, None) == 1        # not a multiple of 16: refused


def test_default_dispatch_reads_no_environment(monkeypatch):
    """The default entry points ignore tuning-looking environment variables;
    overrides reach the library only through the *_tuned calls."""
    shape = (4096, 4096, 4096, 16, 32, 32)
    before = nm.nmspmm_kernel_name(*shape), nm.nmspmm_kernel_name_ws(*shape), nm.nmspmm_workspace_bytes(*shape)
    for key, val in (("TILE", "128x128"), ("SPLITS", "4"), ("KA", "64"), ("GATHER", "1"), ("PS", "1")):
        monkeypatch.setenv("NMSPMM_" + key, val)
    assert (nm.nmspmm_kernel_name(*shape), nm.nmspmm_kernel_name_ws(*shape),
            nm.nmspmm_workspace_bytes(*shape)) == before
    forced = nm.nmspmm_kernel_name(*shape, tuning={"TILE": "128x128", "SPLITS": 4, "KA": 32})
    assert forced.startswith("nm_tiled_kernel<128x128,") and ",ka32," in forced and forced.endswith("split4")


def test_tuning_string_is_checked():
    L = nm.lib()
    shape = (4096, 4096, 4096, 16, 32, 32)
    for bad in (b"FOO=1", b"KA", b"KA=x", b"=3", b"KA=64,,", b"TILE=" + b"x" * 40):
        assert L.nmspmm_kernel_name_tuned(*shape, 0, bad) == b"invalid", bad
        assert L.nmspmm_workspace_bytes_tuned(*shape, bad) == -1, bad
        assert L.nmspmm_run_tuned(0, 0, 0, 0, *shape[:0], 8, 64, 64, 4, 32, 32, ctypes.c_float(1.0), None, 0,
                                  None, 0, bad, None) == nm.NMSPMM_ERR_INVALID_ARG, bad
    assert L.nmspmm_kernel_name_tuned(*shape, 0, b"") == nm.nmspmm_kernel_name(*shape).encode()
    assert L.nmspmm_kernel_name_tuned(*shape, 0, None) == nm.nmspmm_kernel_name(*shape).encode()


def test_noalloc_rejects_shapes_beyond_its_scratch_before_any_gpu_call():
    """nmspmm_run_noalloc checks the shape's workspace against its static
    array before touching the GPU: 128 rows at k = 65536 need a 32 MiB
    transposed A, more than the array's 16 MiB."""
    L = nm.lib()
    assert nm.nmspmm_workspace_bytes(128, 8192, 65536, 4, 32, 64) > nm.NMSPMM_NOALLOC_SCRATCH_BYTES
    st = L.nmspmm_run_noalloc(256, 256, 256, 256, 128, 8192, 65536, 4, 32, 64, ctypes.c_float(1.0), None, 0, None)
    assert st == nm.NMSPMM_ERR_SCRATCH
    assert "scratch" in nm.nmspmm_status_string(st)
    # argument errors come first, and empty products launch nothing
    assert L.nmspmm_run_noalloc(0, 0, 0, 0, 8, 64, 65, 4, 32, 32, ctypes.c_float(1.0), None, 0, None) == \
        nm.NMSPMM_ERR_INVALID_ARG
    assert L.nmspmm_run_noalloc(0, 0, 0, 0, 0, 64, 64, 4, 32, 32, ctypes.c_float(1.0), None, 0, None) == nm.NMSPMM_OK


def test_size_helpers():
    assert nm.nmspmm_bc_elems(4096, 4096, 16, 32) == 2048 * 4096
    assert nm.nmspmm_idx_bytes(4096, 4096, 16, 32, 32) == 2048 * 128
    assert nm.nmspmm_bc_elems(33, 8, 2, 4) == -1
    assert nm.nmspmm_idx_bytes(32, 9, 2, 4, 4) == -1
    assert nm.nmspmm_bc_elems(32, 8, 5, 4) == -1
    assert nm.nmspmm_bc_elems(0, 8, 2, 4) == 0


SHAPES = [
    (64, 96, 4, 32, 32), (256, 256, 16, 32, 32), (128, 128, 8, 32, 64), (48, 30, 3, 8, 3),
    (28, 21, 2, 7, 3), (64, 64, 32, 32, 32), (64, 64, 1, 32, 16), (512, 256, 12, 32, 32),
]


@pytest.mark.parametrize("k,n,N,M,V", SHAPES)
@pytest.mark.parametrize("pruned", [True, False])
def test_compress_matches_oracle_byte_for_byte(k, n, N, M, V, pruned):
    _, Bp, _ = make_inputs(1, k, n, N, M, V, seed=k * 7 + n, dist="normal")
    if not pruned:
        Bp = np.random.default_rng(k + n).standard_normal((k, n)).astype(np.float32)
    Bc, idx = nm.nmspmm_compress(Bp, N, M, V)
    Bc_o, idx_o = oracle.compress(Bp, N, M, V)
    assert np.array_equal(idx, idx_o)
    assert Bc.tobytes() == Bc_o.tobytes()
    assert nm.nmspmm_validate_idx(idx, k, n, N, M, V) == nm.NMSPMM_OK


def test_compress_ties_and_empty():
    Bc, idx = nm.nmspmm_compress(np.ones((8, 4), np.float32), 2, 4, 2)
    assert np.array_equal(idx, np.array([[0, 0], [1, 1], [0, 0], [1, 1]], np.uint8))
    Bc, idx = nm.nmspmm_compress(np.zeros((0, 8), np.float32), 2, 4, 4)
    assert Bc.shape == (0, 8) and idx.shape == (0, 2)


def test_compress_large_uses_threads_and_matches():
    k, n, N, M, V = 2048, 2048, 8, 32, 32
    _, Bp, _ = make_inputs(1, k, n, N, M, V, seed=4)
    Bc, idx = nm.nmspmm_compress(Bp, N, M, V)
    Bc_o, idx_o = oracle.compress(Bp, N, M, V)
    assert np.array_equal(idx, idx_o) and np.array_equal(Bc, Bc_o)


def test_validate_idx_rejects_broken_patterns():
    k, n, N, M, V = 64, 64, 4, 32, 32
    _, Bp, _ = make_inputs(1, k, n, N, M, V, seed=1)
    _, idx = nm.nmspmm_compress(Bp, N, M, V)
    bad = idx.copy()
    bad[2, 1] = 32
    assert nm.nmspmm_validate_idx(bad, k, n, N, M, V) == nm.NMSPMM_ERR_INVALID_ARG
    bad = idx.copy()
    bad[1, 0] = bad[0, 0]
    assert nm.nmspmm_validate_idx(bad, k, n, N, M, V) == nm.NMSPMM_ERR_INVALID_ARG
    bad = idx.copy()
    bad[5, 0], bad[4, 0] = idx[4, 0], idx[5, 0]
    assert nm.nmspmm_validate_idx(bad, k, n, N, M, V) == nm.NMSPMM_ERR_INVALID_ARG
    assert nm.nmspmm_validate_idx(idx, k + 1, n, N, M, V) == nm.NMSPMM_ERR_INVALID_ARG


def test_workspace_bytes():
    """Workspace sizes (host only); -1 for a bad shape.  Short products with V
    a multiple of 32 take the direct-gather kernel: a transposed copy of A
    (k x 16, 32, 64 or 128 floats), the offsets (4 * w * n/V bytes) and, when
    k is split, one partial strip of 32 columns per (strip, split).  Without
    it: one partial tile per (tile, split) of the pipelined streaming kernel,
    0 where the chosen kernel does not split k through a workspace."""
    MiB = 1 << 20
    assert nm.nmspmm_workspace_bytes(64, 8192, 8192, 4, 32, 64) == 2 * MiB + MiB // 2
    assert nm.nmspmm_workspace_bytes(128, 8192, 8192, 4, 32, 64) == 4 * MiB + MiB // 2
    # the variants measured fastest on these shapes
    assert nm.nmspmm_kernel_name_ws(64, 8192, 8192, 4, 32, 64) == "nm_gather_kernel<r64,c32,w8,d4>+prep,split1"
    assert nm.nmspmm_kernel_name_ws(128, 8192, 8192, 4, 32, 64) == "nm_gather_kernel<r128,c32,w4,d4>+prep,split1"
    # forced onto 32 strips of 32 columns, w = 2048: k split 8 ways (8 quads
    # for each of 8 waves)
    gather = {"GATHER": 1}
    assert nm.nmspmm_workspace_bytes(20, 1024, 16384, 4, 32, 64, tuning=gather) == \
        2 * MiB + 16 * 2048 * 4 + 32 * 8 * 32 * 32 * 4
    assert nm.nmspmm_kernel_name_ws(20, 1024, 16384, 4, 32, 64, tuning=gather) == \
        "nm_gather_kernel<r32,c32,w8,d4>+prep,split8"
    # by default strips that do not fill the chip keep the streaming kernels:
    # 4 tiles of 32 x 256, k split 64 ways through the workspace
    assert nm.nmspmm_kernel_name_ws(20, 1024, 16384, 4, 32, 64) == "nm_stream_kernel<r32,c256,bv2,rb16>+ws,split64"
    assert nm.nmspmm_workspace_bytes(20, 1024, 16384, 4, 32, 64) == 4 * 64 * 32 * 256 * 4
    # 16 rows keep the register-operand streaming kernel (atomics, no workspace)
    assert nm.nmspmm_workspace_bytes(16, 8192, 8192, 4, 32, 64) == 0
    assert nm.nmspmm_workspace_bytes(16, 8192, 8192, 4, 32, 64, tuning={"GATHER": 1}) == MiB // 2 + MiB // 2
    assert nm.nmspmm_workspace_bytes(4096, 4096, 4096, 16, 32, 32) == 0    # tiled, no split
    assert nm.nmspmm_workspace_bytes(512, 2048, 2048, 4, 32, 32) == 0      # no split
    assert nm.nmspmm_workspace_bytes(0, 64, 64, 4, 32, 32) == 0
    assert nm.nmspmm_workspace_bytes(10, 64, 65, 4, 32, 32) == -1
    no_gather = {"GATHER": 0}
    # 16 x 8192 x 8192 at 4:32: register-operand streaming kernel, atomics
    assert nm.nmspmm_workspace_bytes(16, 8192, 8192, 4, 32, 64, tuning=no_gather) == 0
    # 64 x 8192 x 8192: pipelined streaming kernel, 64 tiles of 32 x 256, split 4
    assert nm.nmspmm_workspace_bytes(64, 8192, 8192, 4, 32, 64, tuning=no_gather) == 64 * 4 * 32 * 256 * 4
    assert nm.nmspmm_kernel_name_ws(64, 8192, 8192, 4, 32, 64, tuning=no_gather) == \
        "nm_stream_kernel<r32,c256,bv2,rb16>+ws,split4"


def test_run_ws_rejects_misaligned_workspace_before_any_launch():
    L = nm.lib()
    st = L.nmspmm_run_ws(256, 256, 256, 256, 64, 2048, 2048, 4, 32, 64, ctypes.c_float(1.0), None, 0,
                         0x104, 1 << 20, None)
    assert st == nm.NMSPMM_ERR_UNSUPPORTED


def test_dispatch_host_path_without_a_gpu():
    """Every kernel family's host path (plan, argument packing, launch) on a
    machine without a GPU: the launch fails with NMSPMM_ERR_HIP and nothing
    crashes.  (Regression: a general-kernel plan once fell through to the
    tiled launcher.)  Fake device pointers, so this runs only where no GPU is
    visible."""
    torch = pytest.importorskip("torch")
    if torch.cuda.is_available():
        pytest.skip("launches with fake pointers: CPU-only check")
    L = nm.lib()
    shapes = [(17, 24, 10, 3, 8, 2), (300, 320, 320, 16, 32, 32), (129, 128, 96, 4, 32, 16),
              (1100, 96, 1280, 16, 32, 64), (64, 8192, 8192, 4, 32, 64), (16, 4096, 512, 4, 32, 64),
              (20, 16384, 1024, 4, 32, 64)]
    for m, k, n, N, M, V in shapes:
        for ws in (None, 1 << 20):
            st = L.nmspmm_run_ws(4096, 4096, 4096, 8192, m, n, k, N, M, V, ctypes.c_float(1.0), None, 0,
                                 ws, 1 << 30 if ws else 0, None)
            assert st == nm.NMSPMM_ERR_HIP, (m, k, n, N, M, V, st)


@pytest.mark.parametrize("args,status", [
    ((10, 64, 65, 4, 32, 32), nm.NMSPMM_ERR_INVALID_ARG),   # k % M
    ((10, 60, 64, 4, 32, 32), nm.NMSPMM_ERR_INVALID_ARG),   # n % V
    ((10, 64, 64, 0, 32, 32), nm.NMSPMM_ERR_INVALID_ARG),   # N < 1
    ((10, 64, 64, 33, 32, 32), nm.NMSPMM_ERR_INVALID_ARG),  # N > M
    ((10, 512, 512, 4, 512, 32), nm.NMSPMM_ERR_INVALID_ARG),  # M > 256
    ((10, 64, 64, 4, 32, 0), nm.NMSPMM_ERR_INVALID_ARG),    # V < 1
    ((-1, 64, 64, 4, 32, 32), nm.NMSPMM_ERR_INVALID_ARG),   # negative m
    ((0, 64, 64, 4, 32, 32), nm.NMSPMM_OK),                 # m == 0: no launch
    ((10, 0, 64, 4, 32, 32), nm.NMSPMM_OK),                 # n == 0: no launch
])
def test_run_argument_checks_before_any_launch(args, status):
    m, n, k, N, M, V = args
    assert nm.nmspmm_run_ptr(0, 0, 0, 0, m, n, k, N, M, V, 0) == status


def test_run_rejects_null_and_misaligned_pointers():
    # non-empty problem with null buffers: rejected before any HIP call
    assert nm.nmspmm_run_ptr(0, 0, 0, 0, 8, 64, 64, 4, 32, 32, 0) == nm.NMSPMM_ERR_INVALID_ARG
    assert nm.nmspmm_run_ptr(4096, 4096, 4096, 0, 8, 64, 64, 4, 32, 32, 0) == nm.NMSPMM_ERR_INVALID_ARG
    assert nm.nmspmm_run_ptr(4098, 4096, 4096, 4096, 8, 64, 64, 4, 32, 32, 0) == nm.NMSPMM_ERR_UNSUPPORTED
    assert nm.nmspmm_run_ptr(4096, 4096, 4096, 4097, 8, 64, 64, 4, 32, 32, 0) == nm.NMSPMM_ERR_UNSUPPORTED


def test_status_strings():
    assert nm.nmspmm_status_string(0) == "ok"
    assert nm.nmspmm_status_string(1) == "invalid argument"
    assert nm.nmspmm_status_string(3) == "HIP runtime error"
    assert nm.nmspmm_status_string(99) == "unknown status"


def test_kernel_selection():
    assert nm.nmspmm_kernel_name(4096, 4096, 4096, 16, 32, 32).startswith("nm_tiled_kernel<")
    assert nm.nmspmm_kernel_name(5, 12, 8, 1, 4, 1) == "nm_general_kernel"
    assert nm.nmspmm_kernel_name(0, 64, 64, 4, 32, 32) == "none"
    assert nm.nmspmm_kernel_name(8, 64, 65, 4, 32, 32) == "invalid"


def test_run_ex_and_compress_device_argument_checks():
    L = nm.lib()
    # unknown activation, before anything else is looked at
    assert L.nmspmm_run_ex(0, 0, 0, 0, 8, 64, 64, 4, 32, 32, 1.0, None, 7, None) == nm.NMSPMM_ERR_INVALID_ARG
    # empty problem: OK without a launch; misaligned bias: rejected before a launch
    assert L.nmspmm_run_ex(0, 0, 0, 0, 0, 64, 64, 4, 32, 32, 2.0, None, 1, None) == nm.NMSPMM_OK
    assert L.nmspmm_run_ex(4096, 4096, 4096, 4096, 8, 64, 64, 4, 32, 32, 1.0, 4098, 0, None) == \
        nm.NMSPMM_ERR_UNSUPPORTED
    assert L.nmspmm_run_ex(0, 0, 0, 0, 8, 64, 64, 4, 32, 32, 1.0, None, 0, None) == nm.NMSPMM_ERR_INVALID_ARG
    # device packer: shape rules, empty sizes, null and misaligned pointers
    assert L.nmspmm_compress_device(0, 64, 60, 4, 32, 32, 0, 0, None) == nm.NMSPMM_ERR_INVALID_ARG
    assert L.nmspmm_compress_device(0, 0, 64, 4, 32, 32, 0, 0, None) == nm.NMSPMM_OK
    assert L.nmspmm_compress_device(0, 64, 64, 4, 32, 32, 0, 0, None) == nm.NMSPMM_ERR_INVALID_ARG
    assert L.nmspmm_compress_device(4098, 64, 64, 4, 32, 32, 4096, 4096, None) == nm.NMSPMM_ERR_UNSUPPORTED


def test_gather_variant_list_matches_the_source():
    """The GPU tests force every direct-gather instantiation; their list must
    be the source's."""
    src = open(os.path.join(ROOT, "paper_2503_01253_amd", "csrc", "nmspmm_gather.hip")).read()
    block = src[src.index("#define NM_GATHER_CONFIGS(X)"):]
    block = block[:block.index("\n\n")]
    found = [tuple(int(x) for x in t) for t in re.findall(r"X\((\d+), (\d+), (\d+), (\d+)\)", block)]
    gpu = open(os.path.join(ROOT, "tests", "test_gpu_parity.py")).read()
    listed = gpu[gpu.index("\nGATHER_VARIANTS = ["):]
    listed = listed[:listed.index("]\n")]
    tested = [tuple(int(x) for x in t) for t in re.findall(r"\((\d+), (\d+), (\d+), (\d+)\)", listed)]
    assert found and sorted(found) == sorted(tested)


def test_rowgather_variant_list_matches_the_source():
    """The GPU tests force every row-gather instantiation; their list must be
    the source's."""
    src = open(os.path.join(ROOT, "paper_2503_01253_amd", "csrc", "nmspmm_rowgather.hip")).read()
    block = src[src.index("#define NM_ROWGATHER_CONFIGS(X)"):]
    block = block[:block.index("\n\n")]
    found = [tuple(int(x) for x in t) for t in re.findall(r"X\((\d+), (\d+), (\d+), (\d+)\)", block)]
    gpu = open(os.path.join(ROOT, "tests", "test_gpu_parity.py")).read()
    listed = gpu[gpu.index("\nROWGATHER_VARIANTS = ["):]
    listed = listed[:listed.index("]\n")]
    tested = [tuple(int(x) for x in t) for t in re.findall(r"\((\d+), (\d+), (\d+), (\d+)\)", listed)]
    assert found and sorted(found) == sorted(tested)


def test_confusion_argument_checks_without_a_launch():
    """nmspmm_confusion (Eq. 2) refuses bad arguments before any HIP call, and
    an empty matrix is a no-op."""
    L = nm.lib()
    p = 0x1000
    assert L.nmspmm_confusion(p, p, p, -1, 4, None) == nm.NMSPMM_ERR_INVALID_ARG
    assert L.nmspmm_confusion(p, p, p, 4, -1, None) == nm.NMSPMM_ERR_INVALID_ARG
    assert L.nmspmm_confusion(None, None, None, 0, 5, None) == nm.NMSPMM_OK
    assert L.nmspmm_confusion(p, p, p, 7, 0, None) == nm.NMSPMM_OK
    assert L.nmspmm_confusion(None, p, p, 2, 2, None) == nm.NMSPMM_ERR_INVALID_ARG
    assert L.nmspmm_confusion(p, p, None, 2, 2, None) == nm.NMSPMM_ERR_INVALID_ARG
    assert L.nmspmm_confusion(p + 2, p, p, 2, 2, None) == nm.NMSPMM_ERR_UNSUPPORTED
    assert L.nmspmm_confusion(p, p, p, 1 << 40, 1 << 40, None) == nm.NMSPMM_ERR_UNSUPPORTED


def test_run_names_its_workspace_plan():
    """nmspmm_kernel_name names what nmspmm_run launches outside graph
    capture: the direct-gather kernel with its cached workspace where
    nmspmm_kernel_name_ws names it, the kernels that take no workspace
    everywhere else (the tuned query without a workspace)."""
    L = nm.lib()
    for shape in [(64, 8192, 8192, 4, 32, 64), (128, 8192, 8192, 4, 32, 64), (40, 8192, 1536, 4, 32, 64)]:
        assert nm.nmspmm_kernel_name(*shape) == nm.nmspmm_kernel_name_ws(*shape), shape
        assert nm.nmspmm_kernel_name(*shape).startswith("nm_gather_kernel<"), shape
    for shape in [(64, 2048, 4096, 4, 32, 16), (4096, 4096, 4096, 16, 32, 32), (16, 8192, 8192, 4, 32, 64),
                  (1, 8192, 8192, 4, 32, 64)]:
        assert nm.nmspmm_kernel_name(*shape) == L.nmspmm_kernel_name_tuned(*shape, 0, None).decode(), shape
    assert L.nmspmm_kernel_name_tuned(64, 8192, 8192, 4, 32, 64, 0, None).decode() == \
        "nm_stream_kernel<r32,c256,bv2,rb16>+zero,split4"
    # m = 64, n = 2048, k = 4096, V = 16: the pipelined streaming kernel splits
    # k; with a workspace through it, nmspmm_run through atomics
    assert nm.nmspmm_kernel_name_ws(64, 2048, 4096, 4, 32, 16) == "nm_stream_kernel<r32,c128,bv1,rb16>+ws,split8"
    assert nm.nmspmm_kernel_name(64, 2048, 4096, 4, 32, 16) == "nm_stream_kernel<r32,c128,bv1,rb16>+zero,split8"


def test_dispatch_rules_for_short_products():
    """The measured dispatch rules of the short products (host only).
    - Register-operand streaming kernel, k of at most two A chunks: the
      narrowest column tile (down to 32) whose grid stays within 256
      workgroups; a longer k keeps 128 columns and splits k.
    - Up to 128 rows with such a k and a grid that 128 columns would not fill:
      that kernel rather than the pipelined one.
    - The direct-gather kernel only where its strips alone fill the chip.
    - The row-gather kernel for at most 4 rows where its 32-column strips
      alone fill the chip."""
    name = nm.nmspmm_kernel_name
    assert name(256, 256, 256, 16, 32, 32) == "nm_skinny_kernel<c32,bv2,qpw4>,split1"     # 128 workgroups
    assert name(512, 512, 512, 16, 32, 32) == "nm_skinny_kernel<c64,bv2,qpw4>,split1"     # 256
    assert name(512, 512, 512, 32, 32, 32) == "nm_skinny_kernel<c64,bv2,qpw4>,split1"
    assert name(512, 1024, 1024, 16, 32, 32) == "nm_skinny_kernel<c128,bv2,qpw4>,split1"  # 256 at 128
    assert name(256, 512, 1024, 16, 32, 32) == "nm_skinny_kernel<c32,bv2,qpw4>,split1"
    assert name(16, 8192, 1024, 4, 32, 64) == "nm_skinny_kernel<c32,bv2,qpw4>,split1"
    assert name(16, 8192, 8192, 4, 32, 64) == "nm_skinny_kernel<c128,bv4,qpw2>+zero,split4"  # long k
    assert name(64, 2048, 2048, 4, 32, 64) == "nm_skinny_kernel<c32,bv2,qpw4>,split1"
    assert name(128, 2048, 2048, 4, 32, 64) == "nm_skinny_kernel<c64,bv4,qpw4>,split1"
    assert name(64, 2048, 4096, 4, 32, 64).startswith("nm_stream_kernel<")                 # k = 4096
    assert name(512, 512, 512, 4, 32, 32).startswith("nm_stream_kernel<")                   # 512 rows
    ws = nm.nmspmm_kernel_name_ws
    assert ws(64, 8192, 8192, 4, 32, 64).startswith("nm_gather_kernel<")                    # 256 strips
    assert ws(40, 8192, 1536, 4, 32, 64).startswith("nm_gather_kernel<r64,")
    # above 64 rows on short strips (w <= 512, 256 strips): two row halves of 64
    assert ws(128, 8192, 2048, 4, 32, 64) == "nm_gather_kernel<r64x2,c32,w8,d4>+prep,split1"
    assert ws(80, 8192, 2048, 4, 32, 64) == "nm_gather_kernel<r64x2,c32,w8,d4>+prep,split1"
    assert ws(128, 8192, 8192, 4, 32, 64) == "nm_gather_kernel<r128,c32,w4,d4>+prep,split1"     # w = 1024
    assert ws(128, 16384, 4096, 4, 32, 64) == "nm_gather_kernel<r128,c32,w4,d4>+prep,split1"    # 512 strips
    assert ws(128, 8192, 2048, 4, 32, 64, tuning={"GH": 1}) == "nm_gather_kernel<r128,c32,w4,d4>+prep,split1"
    assert ws(128, 4096, 4096, 4, 32, 64).startswith("nm_stream_kernel<")                   # 128 strips
    assert ws(128, 512, 512, 16, 32, 32).startswith("nm_skinny_kernel<c32,")
    assert nm.nmspmm_workspace_bytes(128, 512, 512, 16, 32, 32) == 0
    assert name(1, 8192, 8192, 4, 32, 64) == "nm_rowgather_kernel<r16,c32,w8,d4>,split1"   # 256 strips
    assert name(4, 11008, 4096, 8, 32, 32) == "nm_rowgather_kernel<r16,c32,w8,d4>,split1"
    assert ws(2, 8192, 8192, 4, 32, 64) == "nm_rowgather_kernel<r16,c32,w8,d4>,split1"
    assert nm.nmspmm_workspace_bytes(2, 8192, 8192, 4, 32, 64) == 0
    assert name(8, 8192, 8192, 4, 32, 64).startswith("nm_skinny_kernel<")                  # 8 rows
    assert name(1, 4096, 4096, 8, 32, 32).startswith("nm_skinny_kernel<")                  # 128 strips
    assert name(1, 8192, 8192, 4, 32, 16).startswith("nm_skinny_kernel<")                  # V = 16


def test_dispatch_rules_for_tiled_grids():
    """Host only.  The 16-wave tiles (one workgroup per CU) split k only into
    whole rounds; at N/M <= 1/4 the wide 16-wave tile takes two column
    regions when it needs between one and two rounds and the rest of the
    columns keep at least 160 CUs busy as one round of 128 x 256 tiles (R4)."""
    name = nm.nmspmm_kernel_name
    assert name(1536, 4096, 4096, 8, 32, 32) == "nm_tiled_kernel<128x256m32w16,bv1,ka64,nq4>,split1"   # 192 tiles
    assert name(1536, 4096, 4096, 8, 32, 32, tuning={"TILE": "128x512m32w16"}).endswith("+zero,split2")  # 96
    assert name(2048, 11008, 4096, 8, 32, 32) == (
        "nm_tiled_kernel<128x512m32w16,bv1,ka64,nq4>,split1"
        "+cols8192:nm_tiled_kernel<128x256m32w16,bv1,ka64,nq4>,split1")
    assert "+cols8192:" in name(2048, 11008, 4096, 4, 32, 32)
    assert "+cols" not in name(1536, 11008, 4096, 8, 32, 32)      # 12 tiles left for the second round
    assert "+cols" not in name(2048, 11008, 4096, 16, 32, 32)     # measured slower at 50 %
    assert "+cols" not in name(2048, 11008, 4096, 12, 32, 32)     # and at 62.5 %
    assert "+cols" not in name(4096, 4096, 4096, 8, 32, 32)       # one round
    # a forced tile, stage depth or split keeps one region
    assert "+cols" not in name(2048, 11008, 4096, 8, 32, 32, tuning={"SPLITS": 1})
    assert nm.nmspmm_workspace_bytes(2048, 11008, 4096, 8, 32, 32) == 0
