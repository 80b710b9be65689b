"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bar: every element finite and |C_gpu - C_ref| <= 1e-5 * sum_k |A_ik||B_kj|
(fp32 arithmetic against an fp64 reference), and bit-exact equality on
small-integer inputs whose partial sums are all exact in fp32.
"""
import ctypes
import os
import sys

import numpy as np
import pytest

import oracle
from nm_workloads import RUNS, make_inputs, make_run, table_runs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # the -m gpu suite needs a visible GPU
    pytest.skip("no GPU", allow_module_level=True)

import paper_2503_01253_amd as nm  # noqa: E402


def say(msg):
    print(msg, file=sys.stderr, flush=True)


def to_dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


# Kernel overrides of the current test (the library's tuning entry points:
# forced variants), cleared before every test; empty = the default dispatch.
TUNE = {}


@pytest.fixture(autouse=True)
def _clear_tuning():
    TUNE.clear()
    yield
    TUNE.clear()


def kname(m, n, k, N, M, V):
    return nm.nmspmm_kernel_name(m, n, k, N, M, V, tuning=TUNE)


def kname_ws(m, n, k, N, M, V):
    return nm.nmspmm_kernel_name_ws(m, n, k, N, M, V, tuning=TUNE)


def ws_bytes(m, n, k, N, M, V):
    return nm.nmspmm_workspace_bytes(m, n, k, N, M, V, tuning=TUNE)


def gpu_run(A, Bc, idx, m, n, k, N, M, V, stream=None, fill=float("nan"), workspace=False):
    """Run the library on host arrays; C starts as NaN so unwritten outputs
    fail.  workspace=True: nmspmm_run_ws with a workspace of the size the
    shape takes (the launch the benchmark times)."""
    dA, dBc, didx = to_dev(A), to_dev(Bc), to_dev(idx)
    dC = torch.full((m, n), fill, dtype=torch.float32, device="cuda")
    need = ws_bytes(m, n, k, N, M, V) if workspace else 0
    if need > 0:
        ws = torch.full((need,), 0xFF, dtype=torch.uint8, device="cuda")
        nm.nmspmm_run_ws(dA, dBc, didx, dC, m, n, k, N, M, V, ws, stream=stream, tuning=TUNE)
    else:
        nm.nmspmm_run(dA, dBc, didx, dC, m, n, k, N, M, V, stream=stream, tuning=TUNE)
    torch.cuda.synchronize()
    return dC.cpu().numpy()


def parity(m, k, n, N, M, V, dist, seed):
    say(f"[parity] m={m} k={k} n={n} {N}:{M} V={V} {dist} seed={seed} "
        f"kernel={kname(m, n, k, N, M, V)}")
    A, Bp, _ = make_inputs(m, k, n, N, M, V, seed, dist)
    Bc, idx = nm.nmspmm_compress(Bp, N, M, V)
    Bc_o, idx_o = oracle.compress(Bp, N, M, V)
    assert np.array_equal(idx, idx_o) and np.array_equal(Bc, Bc_o)
    C = gpu_run(A, Bc, idx, m, n, k, N, M, V)
    C_ref = oracle.spmm(A, Bc_o, idx_o, m, n, k, N, M, V)
    Bnd = oracle.bound(A, Bc_o, idx_o, m, n, k, N, M, V)
    return C, C_ref, Bnd


# Shapes that span several tiles and end in ragged tails, over every kernel
# family the dispatcher has (tiled MFMA at V = 16/32/64/128/256, M = 4..32,
# the 62.5% level 12:32, N = M; the general kernel for the rest).
SMALL = [
    (300, 320, 320, 16, 32, 32),
    (300, 256, 448, 8, 32, 64),
    (129, 128, 96, 4, 32, 16),
    (1030, 128, 1088, 4, 32, 32),
    (1100, 96, 1280, 16, 32, 64),
    (65, 64, 64, 32, 32, 32),
    (200, 192, 320, 12, 32, 32),
    (100, 64, 128, 4, 16, 32),
    (64, 48, 128, 4, 16, 32),
    (70, 64, 128, 2, 8, 64),
    (80, 64, 64, 1, 4, 16),
    (70, 64, 256, 8, 32, 128),
    (70, 64, 512, 8, 32, 256),
    (1024, 64, 1024, 8, 32, 512),
    (17, 24, 10, 3, 8, 2),
    (33, 28, 21, 2, 7, 3),
    (5, 64, 64, 1, 32, 32),
    (1, 64, 64, 4, 32, 32),
    (3, 32, 32, 4, 32, 32),
    (20, 256, 512, 20, 32, 32),
    (40, 320, 640, 5, 32, 64),
    (130, 1024, 2048, 4, 32, 64),
    # short products (streaming kernel): ragged column tiles, w not a
    # multiple of 4, wide windows, uneven k splits
    (13, 40, 272, 3, 8, 16),
    (9, 1000, 320, 7, 8, 32),
    (16, 2048, 640, 4, 32, 128),
    (11, 768, 1536, 5, 256, 256),
    (2, 4096, 96, 16, 32, 32),
    (16, 512, 4096, 4, 32, 64),
]


@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("dist", ["uniform", "normal"])
def test_parity_small(shape, dist):
    m, k, n, N, M, V = shape
    C, C_ref, Bnd = parity(m, k, n, N, M, V, dist, seed=m + 3 * k + 7 * n + N)
    r = oracle.check(C, C_ref, Bnd)
    assert r, r


@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "x".join(map(str, s)))
def test_small_integers_exact(shape):
    """With |a|, |b| <= 8 every partial sum is an integer below 2^24, so any
    fp32 summation order gives the exact result: index, gather and tail bugs
    cannot hide inside a tolerance."""
    m, k, n, N, M, V = shape
    C, C_ref, _ = parity(m, k, n, N, M, V, "int", seed=5 + m)
    assert bool(np.array_equal(C.astype(np.float64), C_ref)), \
        f"{int(np.count_nonzero(C.astype(np.float64) != C_ref))} outputs differ"


def full_parity(run, tag):
    """One workload at full size, in the launch the benchmark times (with the
    workspace where the shape takes one): the library's packer must equal the
    oracle's byte for byte, and every output element is compared with the
    oracle's fp64 product at the bar."""
    m, k, n, N, M, V = run.m, run.k, run.n, run.N, run.M, run.V
    say(f"[{tag}] {run.describe()} kernel={kname_ws(m, n, k, N, M, V)}")
    A, Bp, _ = make_run(run)
    Bc, idx = nm.nmspmm_compress(Bp, N, M, V)
    Bc_o, idx_o = oracle.compress(Bp, N, M, V)
    assert np.array_equal(idx, idx_o) and Bc.tobytes() == Bc_o.tobytes()
    C = gpu_run(A, Bc, idx, m, n, k, N, M, V, workspace=True)
    r = oracle.check(C, oracle.spmm(A, Bc_o, idx_o, m, n, k, N, M, V),
                     oracle.bound(A, Bc_o, idx_o, m, n, k, N, M, V))
    say(f"[{tag}] {run.name}: {r}")
    assert r, r


@pytest.mark.parametrize("name", list(RUNS))
def test_parity_full_size(name):
    """Each benchmark workload (256^3 to 4096^3, the MLP shape, the 16-128 row
    decode shapes), every element against the oracle."""
    full_parity(RUNS[name], "full")


TABLE = table_runs()


@pytest.mark.parametrize("name", list(TABLE))
def test_shape_sparsity_table_full(name):
    """Every point of the shape x sparsity sweep (0 % to 87.5 %), every element
    against the oracle."""
    full_parity(TABLE[name], "table")


def test_k_zero_writes_zeros_and_m_zero_is_noop():
    C = gpu_run(np.zeros((40, 0), np.float32), np.zeros((0, 64), np.float32),
                np.zeros((0, 2), np.uint8), 40, 64, 0, 4, 32, 32)
    assert np.all(C == 0)
    dC = torch.full((0, 64), 1.0, device="cuda")
    nm.nmspmm_run(torch.zeros((0, 64), device="cuda"), torch.zeros((8, 64), device="cuda"),
                  torch.zeros((8, 2), dtype=torch.uint8, device="cuda"), dC, 0, 64, 64, 4, 32, 32)
    torch.cuda.synchronize()


def test_deterministic_and_stream_ordered():
    """Without split-k (>= 256 tiles) every output is one workgroup's fixed
    MFMA chain: two runs, on different streams, are bitwise identical."""
    m, k, n, N, M, V = 2048, 128, 8192, 8, 32, 32
    assert kname(m, n, k, N, M, V).endswith(",split1")
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 99)
    Bc, idx = nm.nmspmm_compress(Bp, N, M, V)
    C1 = gpu_run(A, Bc, idx, m, n, k, N, M, V)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        C2 = gpu_run(A, Bc, idx, m, n, k, N, M, V, stream=s)
    same = bool(np.array_equal(C1.view(np.uint32), C2.view(np.uint32)))
    assert same, "two identical launches differ"


def test_split_k_runs_agree_within_tolerance():
    """Split-k adds partial tiles with fp32 atomics, so the summation order
    (and the last bits) may vary between runs; both runs meet the bar."""
    m, k, n, N, M, V = 1030, 256, 1088, 8, 32, 32
    assert "split" in kname(m, n, k, N, M, V)
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 99)
    Bc, idx = nm.nmspmm_compress(Bp, N, M, V)
    C_ref = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    Bnd = oracle.bound(A, Bc, idx, m, n, k, N, M, V)
    for _ in range(2):
        r = oracle.check(gpu_run(A, Bc, idx, m, n, k, N, M, V), C_ref, Bnd)
        assert r, r


@pytest.mark.parametrize("scale", [2.0, 4.0, 8.0])
def test_power_of_two_scaling_is_exact(scale):
    """Eq. 1's M/N factor, applied by the caller to Bc, scales C exactly (one
    workgroup per output tile, so both runs add in the same order)."""
    TUNE["SPLITS"] = "1"
    m, k, n, N, M, V = 300, 256, 320, 32 // int(scale), 32, 32
    assert kname(m, n, k, N, M, V).endswith(",split1")
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 17)
    Bc, idx = nm.nmspmm_compress(Bp, N, M, V)
    C = gpu_run(A, Bc, idx, m, n, k, N, M, V)
    Cs = gpu_run(A, (Bc * np.float32(scale)).astype(np.float32), idx, m, n, k, N, M, V)
    assert bool(np.array_equal(Cs, C * np.float32(scale)))


def test_out_of_range_offsets_stay_in_bounds():
    """An offset >= M is outside the contract; the kernel clamps it, so the
    call completes and writes finite values."""
    m, k, n, N, M, V = 300, 128, 320, 8, 32, 32
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 3)
    Bc, idx = nm.nmspmm_compress(Bp, N, M, V)
    idx = idx.copy()
    idx[::3, ::2] = 255
    C = gpu_run(A, Bc, idx, m, n, k, N, M, V)
    assert np.isfinite(C).all()


TILES = ["256x256", "128x512", "128x128", "64x512", "16x512", "128x256", "256x128",
         "256x256m32", "128x512m32", "128x128m32", "64x512m32", "128x256m32", "64x1024m32",
         "256x256m32w16", "128x512m32w16", "128x256m32w16", "skinny"]
FORCED = [
    (300, 256, 1088, 8, 32, 32),
    (130, 384, 1024, 4, 32, 64),
    (70, 128, 640, 16, 32, 128),
    (200, 96, 576, 12, 32, 64),
    (130, 192, 1024, 32, 32, 64),    # N = M: the 16-wave tiles' stages of 32 rows
    (300, 288, 1088, 16, 32, 32),    # 16:32 at KA = 64 on 128 x 256 (32-row stages), a partial last stage
]


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("shape", FORCED, ids=lambda s: "x".join(map(str, s)))
def test_every_tile_shape_exact(tile, shape):
    """Each tile shape the dispatcher can pick, forced on ragged problems
    with small-integer data (exact in any summation order)."""
    m, k, n, N, M, V = shape
    TUNE["TILE"] = tile
    name = kname(m, n, k, N, M, V)
    if f"<{tile}," not in name and not (tile == "skinny" and name.startswith("nm_skinny")):
        pytest.skip(f"{tile} does not fit {shape} ({name})")
    C, C_ref, _ = parity(m, k, n, N, M, V, "int", seed=7 + m + n)
    assert bool(np.array_equal(C.astype(np.float64), C_ref)), \
        f"{name}: {int(np.count_nonzero(C.astype(np.float64) != C_ref))} outputs differ"


# Deep stages with one A_s slot (the tiles with at most 64 accumulators per
# lane at KA = 128): ragged m / n, a last stage with fewer windows, split-k.
ONE_A_TILES = ["128x256m32", "128x256", "256x128", "128x256m32w16", "128x512m32w16"]
ONE_A = [
    (300, 416, 544, 4, 32, 32),
    (130, 640, 384, 2, 32, 32),
    (260, 384, 288, 4, 32, 32),
]


@pytest.mark.parametrize("splits", [1, 2])
@pytest.mark.parametrize("tile", ONE_A_TILES)
@pytest.mark.parametrize("shape", ONE_A, ids=lambda s: "x".join(map(str, s)))
def test_single_a_slot_deep_stages(tile, shape, splits):
    m, k, n, N, M, V = shape
    TUNE["TILE"] = tile
    TUNE["KA"] = "128"
    TUNE["SPLITS"] = str(splits)
    name = kname(m, n, k, N, M, V)
    if tile in ("128x256m32", "128x256m32w16", "128x512m32w16"):
        assert f"<{tile}," in name and ",ka128," in name, name
    elif f"<{tile}," not in name or ",ka128," not in name:
        pytest.skip(f"{tile} at KA = 128 does not fit {shape} ({name})")
    C, C_ref, _ = parity(m, k, n, N, M, V, "int", seed=11 + m + n)
    assert bool(np.array_equal(C.astype(np.float64), C_ref)), name
    C, C_ref, Bnd = parity(m, k, n, N, M, V, "normal", seed=13 + m + n)
    r = oracle.check(C, C_ref, Bnd)
    assert r, (name, r)


SKINNY = [
    (16, 2048, 640, 4, 32, 64),     # 2 chunks of A per split, ragged column tile
    (13, 3072, 384, 3, 8, 16),      # 3 chunks of 1024 columns, w not a multiple of 4
    (7, 1280, 512, 5, 256, 128),    # M = 256: 4 windows per chunk
    (40, 512, 256, 8, 32, 32),      # several row tiles, rows past m
]


@pytest.mark.parametrize("cols,qpw", [(256, 1), (256, 2), (128, 1), (128, 2), (128, 4),
                                      (64, 1), (64, 2), (64, 4), (64, 8), (32, 1), (32, 2),
                                      (32, 4), (32, 8)])
@pytest.mark.parametrize("splits", [1, 3])
@pytest.mark.parametrize("shape", SKINNY, ids=lambda s: "x".join(map(str, s)))
def test_skinny_variants_exact(shape, splits, cols, qpw):
    """Every streaming-kernel variant (columns per workgroup, quads per wave,
    k split), forced, on small-integer data (exact in any summation order)."""
    m, k, n, N, M, V = shape
    TUNE["TILE"] = "skinny"
    TUNE["PS"] = "0"
    TUNE["SKCOLS"] = str(cols)
    TUNE["QPW"] = str(qpw)
    TUNE["SPLITS"] = str(splits)
    name = kname(m, n, k, N, M, V)
    if not name.startswith(f"nm_skinny_kernel<c{cols},") or f"qpw{qpw}>" not in name:
        pytest.skip(f"variant not instantiated for {shape} ({name})")
    C, C_ref, _ = parity(m, k, n, N, M, V, "int", seed=11 + m + n)
    assert bool(np.array_equal(C.astype(np.float64), C_ref)), \
        f"{name}: {int(np.count_nonzero(C.astype(np.float64) != C_ref))} outputs differ"


# 32-row workgroups (two row tiles share each Bc operand): rows past m in the
# second tile, several chunks, M = 8 and M = 256 windows, split-k
SKINNY32 = [
    (40, 1536, 256, 8, 32, 32),
    (100, 1024, 640, 4, 32, 64),
    (64, 2048, 512, 3, 8, 32),
    (30, 1024, 256, 5, 256, 64),
]


@pytest.mark.parametrize("cols,qpw", [(128, 1), (128, 2), (128, 4), (256, 1), (256, 2)])
@pytest.mark.parametrize("splits", [1, 3])
@pytest.mark.parametrize("shape", SKINNY32, ids=lambda s: "x".join(map(str, s)))
def test_skinny_32_row_variants_exact(shape, splits, cols, qpw):
    """The streaming kernel with 32 rows per workgroup, forced, on
    small-integer data (exact in any summation order), and on normal data
    against the bar."""
    m, k, n, N, M, V = shape
    TUNE["TILE"] = "skinny"
    TUNE["PS"] = "0"
    TUNE["RT"] = "2"
    TUNE["SKCOLS"] = str(cols)
    TUNE["QPW"] = str(qpw)
    TUNE["SPLITS"] = str(splits)
    name = kname(m, n, k, N, M, V)
    if not name.startswith(f"nm_skinny_kernel<c{cols},") or f"qpw{qpw},rows32>" not in name:
        pytest.skip(f"variant not instantiated for {shape} ({name})")
    C, C_ref, _ = parity(m, k, n, N, M, V, "int", seed=21 + m + n)
    assert bool(np.array_equal(C.astype(np.float64), C_ref)), \
        f"{name}: {int(np.count_nonzero(C.astype(np.float64) != C_ref))} outputs differ"
    C, C_ref, Bnd = parity(m, k, n, N, M, V, "normal", seed=23 + m + n)
    r = oracle.check(C, C_ref, Bnd)
    assert r, (name, r)


def test_skinny_32_rows_chosen_for_wide_grids():
    """Without the pipelined kernel, the register-operand streaming kernel
    takes 32-row workgroups where that grid alone fills the chip (512 x 2048
    x 2048 at 4:32), and 16 rows for decode-like shapes."""
    TUNE["PS"] = "0"
    assert kname(512, 2048, 2048, 4, 32, 32).endswith("rows32>,split1")
    assert "rows32" not in kname(64, 8192, 8192, 4, 32, 64)


# ---- pipelined streaming kernel (loader waves, LDS ring) ----
# ragged rows (rows past m in 32- and 64-row tiles), ragged column tiles,
# partial last stages, stages that hold fewer rows than the ring (N = 1, 3,
# 5), M = 8 / 16 / 32 / 64 / 128, V = 16 / 32 / 64, and k splits that leave
# some workgroups without a window
STREAM = [
    (40, 1536, 512, 4, 32, 64),
    (70, 1000, 832, 3, 8, 64),
    (33, 2048, 320, 5, 64, 32),
    (100, 512, 768, 4, 16, 16),
    (16, 4096, 256, 1, 128, 64),
    (20, 64, 256, 4, 32, 64),
]
STREAM_VARIANTS = [(1, 1, 1, 16), (1, 2, 1, 16), (1, 4, 1, 16), (1, 2, 1, 32), (1, 4, 1, 32),
                   (1, 1, 1, 64), (2, 1, 1, 16), (2, 2, 1, 16), (2, 4, 1, 16), (2, 2, 1, 32),
                   (2, 1, 1, 32), (4, 1, 1, 16), (4, 2, 1, 16), (2, 2, 2, 16), (1, 2, 2, 16)]


@pytest.mark.parametrize("splits", [1, 3])
@pytest.mark.parametrize("variant", STREAM_VARIANTS, ids=lambda v: "rt%d_bv%d_cpw%d_rb%d" % v)
@pytest.mark.parametrize("shape", STREAM, ids=lambda s: "x".join(map(str, s)))
def test_stream_variants_exact(shape, variant, splits):
    """Every instantiation of the pipelined streaming kernel (row tiles,
    columns per lane, column groups per wave, ring rows), forced, on
    small-integer data (exact in any summation order) and on normal data
    against the bar."""
    m, k, n, N, M, V = shape
    rt, bv, cpw, rb = variant
    for key, val in (("PS", 1), ("PSRT", rt), ("PSBV", bv), ("PSCPW", cpw), ("PSRB", rb),
                     ("SPLITS", splits)):
        TUNE[key] = str(val)
    name = kname(m, n, k, N, M, V)
    want = "nm_stream_kernel<r%d,c%d,bv%d,rb%d>" % (16 * rt, 128 * bv * cpw, bv, rb)
    if not name.startswith(want):
        pytest.skip(f"variant not available for {shape} ({name})")
    C, C_ref, _ = parity(m, k, n, N, M, V, "int", seed=31 + m + n)
    assert bool(np.array_equal(C.astype(np.float64), C_ref)), \
        f"{name}: {int(np.count_nonzero(C.astype(np.float64) != C_ref))} outputs differ"
    C, C_ref, Bnd = parity(m, k, n, N, M, V, "normal", seed=37 + m + n)
    r = oracle.check(C, C_ref, Bnd)
    assert r, (name, r)


def test_stream_kernel_chosen_by_rule():
    """The dispatcher takes the pipelined kernel for the sparse levels (ring of
    16 or 32 rows) above 16 rows: 32-row tiles with split-k for short
    products, the largest tile that fills the chip for taller ones; and keeps
    the register-operand kernel for 16-row decode shapes and denser levels
    (R5b's shape, whose default with a workspace is the direct-gather kernel:
    the kernels that take none)."""
    TUNE.pop("PS", None)
    assert nm.lib().nmspmm_kernel_name_tuned(64, 8192, 8192, 4, 32, 64, 0, None).decode() == \
        "nm_stream_kernel<r32,c256,bv2,rb16>+zero,split4"
    assert kname(1024, 2048, 2048, 4, 32, 32) == "nm_stream_kernel<r32,c256,bv2,rb16>,split1"
    assert kname(512, 2048, 2048, 8, 32, 32) == "nm_stream_kernel<r16,c256,bv2,rb32>,split1"
    assert kname(512, 512, 512, 4, 32, 32) == "nm_stream_kernel<r16,c128,bv1,rb16>,split1"
    assert kname(16, 8192, 8192, 4, 32, 64).startswith("nm_skinny_kernel")
    assert kname(512, 1024, 1024, 16, 32, 32).startswith("nm_skinny_kernel")
    TUNE["PS"] = "0"
    assert kname(64, 8192, 8192, 4, 32, 64).startswith("nm_skinny_kernel")


def test_dense_comparator_is_true_fp32():
    """The benchmark's dense comparator (torch.matmul on the decompressed B,
    TF32 off) meets the same bar, so it is a true fp32 GEMM."""
    torch.backends.cuda.matmul.allow_tf32 = False
    torch.set_float32_matmul_precision("highest")
    m, k, n, N, M, V = 256, 2048, 512, 16, 32, 32
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 21)
    Bc, idx = oracle.compress(Bp, N, M, V)
    C = torch.matmul(to_dev(A), to_dev(Bp)).cpu().numpy()
    r = oracle.check(C, oracle.spmm(A, Bc, idx, m, n, k, N, M, V), oracle.bound(A, Bc, idx, m, n, k, N, M, V))
    assert r, r


# ---- output epilogue (nmspmm_run_ex) ----
# one shape per kernel family: tiled (one workgroup per tile), tiled split-k,
# streaming, streaming split-k, general kernel
EPI_SHAPES = [
    (2048, 128, 8192, 8, 32, 32),
    (64, 4096, 2048, 4, 32, 64),     # pipelined streaming kernel, split-k
    (8100, 160, 2784, 8, 32, 32),    # the tiled kernel over two column regions
    (512, 512, 512, 4, 32, 32),      # pipelined streaming kernel, fused epilogue
    (300, 256, 1088, 8, 32, 32),
    (16, 2048, 640, 4, 32, 128),
    (16, 512, 4096, 4, 32, 64),
    (17, 24, 10, 3, 8, 2),
]


# The tiled kernel over two column regions (one round of whole 128 x 512
# 16-wave tiles, then the rest as one round of 128 x 256 ones): rows past m,
# a ragged last column tile, a partial last stage, V = 64.
TWO_REGIONS = [(8100, 160, 2784, 8, 32, 32), (8192, 128, 2752, 4, 32, 64), (8192, 96, 2816, 8, 32, 32)]


@pytest.mark.parametrize("shape", TWO_REGIONS, ids=lambda s: "x".join(map(str, s)))
def test_two_column_regions_exact(shape):
    m, k, n, N, M, V = shape
    name = kname(m, n, k, N, M, V)
    assert "+cols2048:nm_tiled_kernel<128x256m32w16," in name and name.startswith("nm_tiled_kernel<128x512m32w16,")
    C, C_ref, _ = parity(m, k, n, N, M, V, "int", seed=7 + n)
    assert bool(np.array_equal(C.astype(np.float64), C_ref)), \
        f"{name}: {int(np.count_nonzero(C.astype(np.float64) != C_ref))} outputs differ"


def run_ex(A, Bc, idx, m, n, k, N, M, V, alpha, bias, act):
    dC = torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")
    nm.nmspmm_run_ex(to_dev(A), to_dev(Bc), to_dev(idx), dC, m, n, k, N, M, V, alpha=alpha,
                     bias=None if bias is None else to_dev(bias), act=act, tuning=TUNE)
    torch.cuda.synchronize()
    return dC.cpu().numpy()


@pytest.mark.parametrize("act", ["none", "relu", "gelu"])
@pytest.mark.parametrize("shape", EPI_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_run_ex_epilogue(shape, act):
    """act(alpha * C + bias) against the oracle's epilogue on its fp64 product;
    alpha = M/N (Eq. 1's factor).  Bound: the product's bar propagated through
    alpha and the activation (|d act| <= 1.13 |d y|), plus fp32 rounding of the
    epilogue itself."""
    m, k, n, N, M, V = shape
    say(f"[epilogue] {shape} {act} kernel={kname(m, n, k, N, M, V)}")
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 40 + m, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    bias = np.random.default_rng(m).standard_normal(n).astype(np.float32)
    alpha = M / N
    C_ref = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    Bnd = oracle.bound(A, Bc, idx, m, n, k, N, M, V)
    Y_ref = oracle.epilogue(C_ref, alpha, bias, act)
    y_ref = oracle.epilogue(C_ref, alpha, bias, "none")
    Y = run_ex(A, Bc, idx, m, n, k, N, M, V, alpha, bias, act).astype(np.float64)
    tol = (1.2 * (alpha * 1e-5 * Bnd + 2.0 ** -22 * (np.abs(alpha * C_ref) + np.abs(bias)))
           + 4e-7 * (np.abs(y_ref) + np.abs(Y_ref)) + 1e-30)
    err = np.abs(Y - Y_ref)
    assert np.isfinite(Y).all()
    assert bool((err <= tol).all()), f"worst err/tol {float((err / tol).max()):.3g}"


@pytest.mark.parametrize("shape", EPI_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_run_ex_exact_on_integers(shape):
    """Small integers, a power-of-two alpha and an integer bias: every value is
    exact in fp32, so the epilogue must match the oracle bit for bit."""
    m, k, n, N, M, V = shape
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 3 + m, "int")
    Bc, idx = oracle.compress(Bp, N, M, V)
    bias = np.random.default_rng(n).integers(-50, 50, n).astype(np.float32)
    C_ref = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    for alpha, act in ((4.0, "relu"), (0.5, "none")):
        Y = run_ex(A, Bc, idx, m, n, k, N, M, V, alpha, bias, act)
        assert bool(np.array_equal(Y.astype(np.float64), oracle.epilogue(C_ref, alpha, bias, act)))


def test_run_ex_trivial_epilogue_is_nmspmm_run():
    m, k, n, N, M, V = 2048, 128, 8192, 8, 32, 32
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 12)
    Bc, idx = nm.nmspmm_compress(Bp, N, M, V)
    C = gpu_run(A, Bc, idx, m, n, k, N, M, V)
    Y = run_ex(A, Bc, idx, m, n, k, N, M, V, 1.0, None, "none")
    assert bool(np.array_equal(C.view(np.uint32), Y.view(np.uint32)))


# ---- split-k through a caller-provided workspace (nmspmm_run_ws) ----
# the pipelined streaming kernel at 16, 32 and 64 rows, ragged tiles, V = 16,
# and a split that gets no window of k
WS_CASES = [
    ((100, 512, 768, 2, 16, 16), {"PS": "1", "PSRT": "1", "SPLITS": "3"}),
    ((40, 1536, 512, 4, 32, 64), {"PS": "1", "PSRT": "2", "SPLITS": "3"}),
    ((70, 1536, 832, 4, 32, 64), {"PS": "1", "PSRT": "4", "SPLITS": "5"}),
    ((20, 160, 256, 4, 32, 64), {"PS": "1", "PSRT": "1", "SPLITS": "4"}),   # 5 windows: split 3 gets none
]


def new_workspace(m, n, k, N, M, V):
    need = ws_bytes(m, n, k, N, M, V)
    assert need > 0
    ws = torch.full((need,), 0xFF, dtype=torch.uint8, device="cuda")   # contents irrelevant (NaN bytes)
    assert ws.data_ptr() % 256 == 0
    return ws


def run_ws(A, Bc, idx, m, n, k, N, M, V, ws, alpha=1.0, bias=None, act="none"):
    dC = torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")
    nm.nmspmm_run_ws(to_dev(A), to_dev(Bc), to_dev(idx), dC, m, n, k, N, M, V, ws, alpha=alpha,
                     bias=None if bias is None else to_dev(bias), act=act, tuning=TUNE)
    torch.cuda.synchronize()
    return dC.cpu().numpy()


@pytest.mark.parametrize("shape,env", WS_CASES, ids=["rows16_v16", "rows32", "rows64", "rows16_empty_split"])
def test_run_ws_split_k(shape, env):
    """Split-k through the workspace: bit-exact on small integers (twice in a
    row on one workspace), the epilogue applied once and exactly, normal data
    within the bar and bit-identical between runs."""
    for key, val in env.items():
        TUNE[key] = val
    TUNE["GATHER"] = "0"
    m, k, n, N, M, V = shape
    name = kname_ws(m, n, k, N, M, V)
    say(f"[workspace] {shape} {name}")
    assert "+ws,split" in name
    ws = new_workspace(m, n, k, N, M, V)
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 5 + m, "int")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C_ref = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    for _ in range(2):
        C = run_ws(A, Bc, idx, m, n, k, N, M, V, ws)
        assert bool(np.array_equal(C.astype(np.float64), C_ref))
    bias = np.random.default_rng(n).integers(-50, 50, n).astype(np.float32)
    Y = run_ws(A, Bc, idx, m, n, k, N, M, V, ws, alpha=4.0, bias=bias, act="relu")
    assert bool(np.array_equal(Y.astype(np.float64), oracle.epilogue(C_ref, 4.0, bias, "relu")))
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 9 + m, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C1 = run_ws(A, Bc, idx, m, n, k, N, M, V, ws)
    C2 = run_ws(A, Bc, idx, m, n, k, N, M, V, ws)
    assert bool(np.array_equal(C1.view(np.uint32), C2.view(np.uint32)))
    r = oracle.check(C1, oracle.spmm(A, Bc, idx, m, n, k, N, M, V), oracle.bound(A, Bc, idx, m, n, k, N, M, V))
    assert r, (name, r)


def test_run_ws_small_or_missing_workspace_runs_as_run_ex():
    """A workspace smaller than needed, or none, leaves the call to the atomic
    path of nmspmm_run_ex (within the bar)."""
    m, k, n, N, M, V = 64, 2048, 2048, 4, 32, 64
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 77, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C_ref = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    Bnd = oracle.bound(A, Bc, idx, m, n, k, N, M, V)
    small = torch.zeros(256, dtype=torch.uint8, device="cuda")
    for ws in (small, None):
        C = run_ws(A, Bc, idx, m, n, k, N, M, V, ws)
        assert oracle.check(C, C_ref, Bnd)
    assert int(small.to(torch.int64).sum()) == 0   # untouched


@pytest.mark.parametrize("gather", ["0", "1"])
def test_run_ws_graph_replay(gather):
    """nmspmm_run_ws captured in a HIP graph (two kernels, no fill of C and no
    memset: split-k of the pipelined streaming kernel, or the transposition
    pass and the direct-gather kernel): every replay, with eager work between
    replays, gives the eager result bit for bit."""
    TUNE["GATHER"] = gather
    m, k, n, N, M, V = 64, 4096, 2048, 4, 32, 64
    name = kname_ws(m, n, k, N, M, V)
    say(f"[graph] {name}")
    assert ("+ws,split" if gather == "0" else "nm_gather_kernel") in name
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 78, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    dA, dBc, didx = to_dev(A), to_dev(Bc), to_dev(idx)
    ws = new_workspace(m, n, k, N, M, V)
    dC = torch.empty((m, n), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        nm.nmspmm_run_ws(dA, dBc, didx, dC, m, n, k, N, M, V, ws, tuning=TUNE)
    torch.cuda.synchronize()
    eager = dC.cpu().numpy().copy()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        nm.nmspmm_run_ws(dA, dBc, didx, dC, m, n, k, N, M, V, ws, tuning=TUNE)
    for i in range(3):
        dC.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert bool(np.array_equal(dC.cpu().numpy().view(np.uint32), eager.view(np.uint32))), f"replay {i}"


# ---- cached workspaces of nmspmm_run / nmspmm_run_ex ----
CACHED_WS_SHAPES = [
    (64, 8192, 8192, 4, 32, 64),    # R5b
    (128, 2048, 8192, 4, 32, 64),   # 128 rows
    (40, 1536, 8192, 4, 32, 64),    # 40 rows in the 64-row variant
]


@pytest.mark.parametrize("shape", CACHED_WS_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_run_takes_cached_workspace(shape):
    """Outside graph capture nmspmm_run and nmspmm_run_ex take the direct-
    gather kernel with the workspace the library keeps for the stream where
    nmspmm_run_ws would run it: the name is that of nmspmm_kernel_name_ws, and
    the output is bit-identical to nmspmm_run_ws's (with and without the
    epilogue), twice in a row, and within the bar."""
    m, k, n, N, M, V = shape
    name = nm.nmspmm_kernel_name(m, n, k, N, M, V)
    say(f"[cached ws] {shape} {name}")
    assert name == nm.nmspmm_kernel_name_ws(m, n, k, N, M, V)
    assert name.startswith("nm_gather_kernel<")
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 51 + m, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    dA, dBc, didx = to_dev(A), to_dev(Bc), to_dev(idx)
    ws = new_workspace(m, n, k, N, M, V)
    bias = torch.randn(n, device="cuda")
    for kw in ({}, {"alpha": M / N, "bias": bias, "act": "gelu"}):
        ref = torch.full((m, n), float("nan"), device="cuda")
        nm.nmspmm_run_ws(dA, dBc, didx, ref, m, n, k, N, M, V, ws, **kw)
        for _ in range(2):
            out = torch.full((m, n), float("nan"), device="cuda")
            if kw:
                nm.nmspmm_run_ex(dA, dBc, didx, out, m, n, k, N, M, V, **kw)
            else:
                nm.nmspmm_run(dA, dBc, didx, out, m, n, k, N, M, V)
            torch.cuda.synchronize()
            assert torch.equal(out.view(torch.int32), ref.view(torch.int32))
    out = torch.full((m, n), float("nan"), device="cuda")
    nm.nmspmm_run(dA, dBc, didx, out, m, n, k, N, M, V)
    torch.cuda.synchronize()
    r = oracle.check(out.cpu().numpy(), oracle.spmm(A, Bc, idx, m, n, k, N, M, V),
                     oracle.bound(A, Bc, idx, m, n, k, N, M, V))
    assert r, (name, r)


def test_run_under_capture_takes_no_workspace():
    """Captured into a HIP graph, nmspmm_run allocates nothing: it records the
    kernels that take no workspace (split-k with a fill kernel and atomics),
    and every replay, with eager work between replays, meets the bar."""
    m, k, n, N, M, V = 64, 4096, 8192, 4, 32, 64
    no_ws = nm.lib().nmspmm_kernel_name_tuned(m, n, k, N, M, V, 0, None).decode()
    say(f"[capture] {nm.nmspmm_kernel_name(m, n, k, N, M, V)} / under capture {no_ws}")
    assert "+prep" not in no_ws and "+ws" not in no_ws
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 61, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    dA, dBc, didx = to_dev(A), to_dev(Bc), to_dev(idx)
    C_ref = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    Bnd = oracle.bound(A, Bc, idx, m, n, k, N, M, V)
    dC = torch.empty((m, n), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        nm.nmspmm_run(dA, dBc, didx, dC, m, n, k, N, M, V)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        nm.nmspmm_run(dA, dBc, didx, dC, m, n, k, N, M, V)
    for i in range(3):
        dC.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert oracle.check(dC.cpu().numpy(), C_ref, Bnd), f"replay {i}"
        eager = torch.full((m, n), float("nan"), device="cuda")
        nm.nmspmm_run(dA, dBc, didx, eager, m, n, k, N, M, V)
        torch.cuda.synchronize()
        assert oracle.check(eager.cpu().numpy(), C_ref, Bnd)


def test_run_cached_workspaces_on_two_streams():
    """Calls on two streams at once each take their own cached workspace: both
    outputs bit-identical to nmspmm_run_ws's."""
    m, k, n, N, M, V = 64, 8192, 8192, 4, 32, 64
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 71, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    dA, dBc, didx = to_dev(A), to_dev(Bc), to_dev(idx)
    A2 = torch.randn((m, k), device="cuda")
    ref = [torch.empty((m, n), device="cuda") for _ in range(2)]
    ws = new_workspace(m, n, k, N, M, V)
    for a, r in zip((dA, A2), ref):
        nm.nmspmm_run_ws(a, dBc, didx, r, m, n, k, N, M, V, ws)
    torch.cuda.synchronize()
    outs = [torch.full((m, n), float("nan"), device="cuda") for _ in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for _ in range(3):
        for a, o, st in zip((dA, A2), outs, streams):
            with torch.cuda.stream(st):
                nm.nmspmm_run(a, dBc, didx, o, m, n, k, N, M, V, stream=st)
        torch.cuda.synchronize()
        for o, r in zip(outs, ref):
            assert torch.equal(o.view(torch.int32), r.view(torch.int32))


def test_run_cached_workspace_on_a_reused_stream_handle():
    """HIP hands a new stream the handle of the stream destroyed just before;
    the workspace cached for that handle is then ordered after the destroyed
    stream's last kernels, which are still running when the new stream's
    call is enqueued.  Both outputs bit-identical to nmspmm_run_ws's."""
    hip = ctypes.CDLL(os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so"))
    m, k, n, N, M, V = 128, 2048, 8192, 4, 32, 64
    assert nm.nmspmm_kernel_name(m, n, k, N, M, V).startswith("nm_gather_kernel<")
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 73, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    dA, dBc, didx = to_dev(A), to_dev(Bc), to_dev(idx)
    A2 = torch.randn((m, k), device="cuda")
    ref = [torch.empty((m, n), device="cuda") for _ in range(2)]
    ws = new_workspace(m, n, k, N, M, V)
    for a, r in zip((dA, A2), ref):
        nm.nmspmm_run_ws(a, dBc, didx, r, m, n, k, N, M, V, ws)
    torch.cuda.synchronize()
    reused = 0
    for _ in range(3):
        outs = [torch.full((m, n), float("nan"), device="cuda") for _ in range(2)]
        torch.cuda.synchronize()
        handles = []
        for a, o in zip((dA, A2), outs):
            h = ctypes.c_void_p()
            assert hip.hipStreamCreate(ctypes.byref(h)) == 0
            handles.append(h.value)
            st = torch.cuda.ExternalStream(h.value)
            for _ in range(4):   # a queue of work still running at the destroy
                nm.nmspmm_run(a, dBc, didx, o, m, n, k, N, M, V, stream=st)
            assert hip.hipStreamDestroy(h) == 0
        reused += handles[0] == handles[1]
        torch.cuda.synchronize()
        for o, r in zip(outs, ref):
            assert torch.equal(o.view(torch.int32), r.view(torch.int32))
    say(f"[cached ws] reused stream handles: {reused} of 3")


def test_run_cached_workspaces_past_the_cap_and_from_threads():
    """More streams than the library keeps buffers for (each new one
    releases the least recently used idle buffer after its last kernels),
    then four host threads calling at once on their own streams: every
    output bit-identical to nmspmm_run_ws's."""
    import threading
    m, k, n, N, M, V = 64, 2048, 8192, 4, 32, 64
    assert nm.nmspmm_kernel_name(m, n, k, N, M, V).startswith("nm_gather_kernel<")
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 79, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    dA, dBc, didx = to_dev(A), to_dev(Bc), to_dev(idx)
    ref = torch.empty((m, n), device="cuda")
    nm.nmspmm_run_ws(dA, dBc, didx, ref, m, n, k, N, M, V, new_workspace(m, n, k, N, M, V))
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(20)]
    outs = [torch.full((m, n), float("nan"), device="cuda") for _ in streams]
    for st, o in zip(streams, outs):
        for _ in range(2):
            nm.nmspmm_run(dA, dBc, didx, o, m, n, k, N, M, V, stream=st)
    torch.cuda.synchronize()
    for o in outs:
        assert torch.equal(o.view(torch.int32), ref.view(torch.int32))
    errors = []

    def worker(st, o):
        try:
            with torch.cuda.stream(st):
                for _ in range(10):
                    nm.nmspmm_run(dA, dBc, didx, o, m, n, k, N, M, V, stream=st)
            st.synchronize()
        except Exception as e:   # reported by the main thread
            errors.append(e)

    outs = [torch.full((m, n), float("nan"), device="cuda") for _ in range(4)]
    torch.cuda.synchronize()
    threads = [threading.Thread(target=worker, args=(streams[i], outs[i])) for i in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    torch.cuda.synchronize()
    for o in outs:
        assert torch.equal(o.view(torch.int32), ref.view(torch.int32))


# ---- direct-gather kernel (nmspmm_run_ws on short products) ----
GATHER_SHAPES = [
    (1, 512, 256, 4, 32, 32),       # one row
    (5, 1024, 512, 2, 4, 32),
    (16, 2048, 1024, 4, 32, 64),
    (17, 776, 320, 3, 8, 32),       # w = 291: ragged last quad
    (40, 1536, 512, 4, 32, 64),
    (64, 1000, 512, 5, 8, 64),      # w = 625
    (100, 832, 768, 1, 8, 128),     # w = 104, four strips per column block
    (128, 2048, 1024, 16, 32, 32),  # 50 %
    (128, 96, 64, 8, 32, 32),       # w = 24: one to two quads per wave
    (33, 32, 256, 4, 32, 32),       # one window: most waves get no quad
    (70, 2040, 96, 3, 8, 32),       # w = 765, three strips
]


@pytest.mark.parametrize("splits", ["auto", "3"])
@pytest.mark.parametrize("shape", GATHER_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_gather_kernel_exact(shape, splits):
    """The direct-gather kernel (forced), with and without split-k: bit-exact on
    small integers twice in a row on one workspace, the epilogue applied once
    and exactly, normal data within the bar and bit-identical between runs."""
    TUNE["GATHER"] = "1"
    if splits != "auto":
        TUNE["SPLITS"] = splits
    m, k, n, N, M, V = shape
    name = kname_ws(m, n, k, N, M, V)
    say(f"[gather] {shape} {name}")
    rows = 16 if m <= 16 else 32 if m <= 32 else 64 if m <= 64 else 128
    # above 64 rows without split-k on short strips: two row halves of 64
    assert name.startswith(("nm_gather_kernel<r%d," % rows,) + (("nm_gather_kernel<r64x2,",) if m > 64 else ()))
    w = k // M * N
    if splits != "auto" and (w + 3) // 4 >= 3:
        assert name.endswith(",split3")
    ws = new_workspace(m, n, k, N, M, V)
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 11 + m, "int")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C_ref = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    for _ in range(2):
        C = run_ws(A, Bc, idx, m, n, k, N, M, V, ws)
        assert bool(np.array_equal(C.astype(np.float64), C_ref)), \
            f"{int(np.count_nonzero(C.astype(np.float64) != C_ref))} outputs differ"
    bias = np.random.default_rng(n).integers(-50, 50, n).astype(np.float32)
    Y = run_ws(A, Bc, idx, m, n, k, N, M, V, ws, alpha=4.0, bias=bias, act="relu")
    assert bool(np.array_equal(Y.astype(np.float64), oracle.epilogue(C_ref, 4.0, bias, "relu")))
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 13 + m, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C1 = run_ws(A, Bc, idx, m, n, k, N, M, V, ws)
    C2 = run_ws(A, Bc, idx, m, n, k, N, M, V, ws)
    assert bool(np.array_equal(C1.view(np.uint32), C2.view(np.uint32)))
    r = oracle.check(C1, oracle.spmm(A, Bc, idx, m, n, k, N, M, V), oracle.bound(A, Bc, idx, m, n, k, N, M, V))
    assert r, (name, r)


# every instantiated variant {RT, CT, NW, D}; tests/test_abi.py checks this list against the source
GATHER_VARIANTS = [
    (1, 2, 8, 4), (1, 2, 8, 8), (1, 4, 8, 4), (1, 4, 4, 8),
    (2, 2, 8, 4), (2, 2, 8, 8), (2, 4, 8, 4),
    (4, 2, 8, 4), (4, 2, 8, 3), (4, 2, 8, 8), (4, 4, 8, 4), (4, 4, 4, 8),
    (8, 2, 4, 4), (8, 2, 4, 8), (8, 2, 8, 4), (8, 4, 4, 4), (8, 4, 4, 6),
]
# per row-tile count: a ragged shape (w not a multiple of 4 where N allows) with V a multiple of 64
GATHER_VARIANT_SHAPES = {1: (9, 1024, 512, 4, 32, 64), 2: (30, 776, 384, 3, 8, 64),
                         4: (50, 1000, 512, 5, 8, 64), 8: (100, 832, 768, 1, 8, 128)}


@pytest.mark.parametrize("splits", [1, 3])
@pytest.mark.parametrize("variant", GATHER_VARIANTS, ids=lambda v: "rt%d_ct%d_nw%d_d%d" % v)
def test_gather_variants_exact(variant, splits):
    """Every direct-gather instantiation, forced, with and without split-k:
    bit-exact on small integers and within the bar on normal data."""
    rt, ct, nw, d = variant
    for key, val in (("GATHER", 1), ("GCT", ct), ("GNW", nw), ("GD", d), ("SPLITS", splits)):
        TUNE[key] = str(val)
    m, k, n, N, M, V = GATHER_VARIANT_SHAPES[rt]
    name = kname_ws(m, n, k, N, M, V)
    say(f"[gather variant] {variant} split{splits} {name}")
    assert name == f"nm_gather_kernel<r{16 * rt},c{16 * ct},w{nw},d{d}>+prep,split{splits}"
    ws = new_workspace(m, n, k, N, M, V)
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 31 + m, "int")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C = run_ws(A, Bc, idx, m, n, k, N, M, V, ws)
    assert bool(np.array_equal(C.astype(np.float64), oracle.spmm(A, Bc, idx, m, n, k, N, M, V)))
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 37 + m, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C = run_ws(A, Bc, idx, m, n, k, N, M, V, ws)
    r = oracle.check(C, oracle.spmm(A, Bc, idx, m, n, k, N, M, V), oracle.bound(A, Bc, idx, m, n, k, N, M, V))
    assert r, (name, r)


@pytest.mark.parametrize("shape", [(65, 1024, 512, 4, 32, 64), (100, 832, 768, 1, 8, 128), (128, 2048, 1024, 16, 32, 32),
                                   (97, 776, 320, 3, 8, 32)], ids=lambda s: "x".join(map(str, s)))
def test_gather_row_halves_exact(shape):
    """Above 64 rows, the direct-gather kernel forced into two row halves of
    64 rows (each half its own workgroup and At; the second half ragged):
    bit-exact on small integers twice in a row on one workspace, the epilogue
    applied once, normal data within the bar."""
    TUNE.update({"GATHER": "1", "SPLITS": "1", "GH": "2"})
    m, k, n, N, M, V = shape
    name = kname_ws(m, n, k, N, M, V)
    say(f"[gather halves] {shape} {name}")
    assert name.startswith("nm_gather_kernel<r64x2,")
    ws = new_workspace(m, n, k, N, M, V)
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 17 + m, "int")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C_ref = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    for _ in range(2):
        C = run_ws(A, Bc, idx, m, n, k, N, M, V, ws)
        assert bool(np.array_equal(C.astype(np.float64), C_ref)), \
            f"{int(np.count_nonzero(C.astype(np.float64) != C_ref))} outputs differ"
    bias = np.random.default_rng(n).integers(-50, 50, n).astype(np.float32)
    Y = run_ws(A, Bc, idx, m, n, k, N, M, V, ws, alpha=4.0, bias=bias, act="relu")
    assert bool(np.array_equal(Y.astype(np.float64), oracle.epilogue(C_ref, 4.0, bias, "relu")))
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 19 + m, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C = run_ws(A, Bc, idx, m, n, k, N, M, V, ws)
    r = oracle.check(C, oracle.spmm(A, Bc, idx, m, n, k, N, M, V), oracle.bound(A, Bc, idx, m, n, k, N, M, V))
    assert r, (name, r)


def test_gather_kernel_reused_workspace_smaller_shape():
    """One workspace, a large call then a smaller one of another row count: the
    second call's transposed copy and offsets replace the first's."""
    TUNE["GATHER"] = "1"
    big, small = (128, 2048, 1024, 4, 32, 32), (20, 1024, 512, 4, 32, 64)
    ws = new_workspace(*[big[i] for i in (0, 2, 1, 3, 4, 5)])
    assert ws.numel() >= ws_bytes(*[small[i] for i in (0, 2, 1, 3, 4, 5)])
    for m, k, n, N, M, V in (big, small):
        A, Bp, _ = make_inputs(m, k, n, N, M, V, 21 + m, "int")
        Bc, idx = oracle.compress(Bp, N, M, V)
        C = run_ws(A, Bc, idx, m, n, k, N, M, V, ws)
        assert bool(np.array_equal(C.astype(np.float64), oracle.spmm(A, Bc, idx, m, n, k, N, M, V)))


def test_gather_kernel_chosen_by_rule():
    """With a workspace, the 64- and 128-row products of the benchmark take
    the direct-gather kernel; 16 rows, V = 16 and tall products do not."""
    assert kname_ws(64, 8192, 8192, 4, 32, 64).startswith("nm_gather_kernel<r64,c32,")
    assert kname_ws(128, 8192, 8192, 4, 32, 64).startswith("nm_gather_kernel<r128,c32,")
    assert not kname_ws(16, 8192, 8192, 4, 32, 64).startswith("nm_gather")
    assert not kname_ws(64, 2048, 2048, 4, 32, 16).startswith("nm_gather")
    assert not kname_ws(4096, 4096, 4096, 16, 32, 32).startswith("nm_gather")


# ---- row-gather kernel (one launch, at most 32 rows) ----
ROWGATHER_SHAPES = [
    (1, 512, 256, 4, 32, 32),        # one row
    (5, 1024, 512, 2, 4, 32),        # M = 4: eight windows per A line
    (16, 2048, 1024, 4, 32, 64),
    (16, 776, 512, 3, 8, 32),        # w = 291: ragged last quad, quads span windows
    (9, 1000, 512, 5, 8, 64),        # w = 625
    (17, 4096, 2048, 1, 32, 64),     # N = 1 (no window division), 17 rows: two row tiles
    (32, 2048, 1024, 16, 32, 32),    # 50 %, 32 rows
    (20, 96, 128, 8, 32, 32),        # w = 24: six quads for eight waves
    (12, 32, 256, 4, 32, 32),        # one window: one quad in all
    (30, 256, 128, 32, 32, 32),      # N = M
    (3, 2048, 256, 2, 32, 128),      # four strips per column block
]


def run_plain(A, Bc, idx, m, n, k, N, M, V, alpha=1.0, bias=None, act="none"):
    dC = torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")
    nm.nmspmm_run_ex(to_dev(A), to_dev(Bc), to_dev(idx), dC, m, n, k, N, M, V, alpha=alpha,
                     bias=None if bias is None else to_dev(bias), act=act, tuning=TUNE)
    torch.cuda.synchronize()
    return dC.cpu().numpy()


@pytest.mark.parametrize("shape", ROWGATHER_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_rowgather_kernel_exact(shape):
    """The row-gather kernel (forced): bit-exact on small integers, the
    epilogue applied once and exactly, normal data within the bar and
    bit-identical between runs."""
    TUNE["RG"] = "1"
    m, k, n, N, M, V = shape
    name = kname(m, n, k, N, M, V)
    say(f"[rowgather] {shape} {name}")
    assert name.startswith("nm_rowgather_kernel<r%d," % (16 if m <= 16 else 32)), name
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 41 + m, "int")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C_ref = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    C = run_plain(A, Bc, idx, m, n, k, N, M, V)
    assert bool(np.array_equal(C.astype(np.float64), C_ref)), \
        f"{int(np.count_nonzero(C.astype(np.float64) != C_ref))} outputs differ"
    bias = np.random.default_rng(n).integers(-50, 50, n).astype(np.float32)
    Y = run_plain(A, Bc, idx, m, n, k, N, M, V, alpha=4.0, bias=bias, act="relu")
    assert bool(np.array_equal(Y.astype(np.float64), oracle.epilogue(C_ref, 4.0, bias, "relu")))
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 43 + m, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C1 = run_plain(A, Bc, idx, m, n, k, N, M, V)
    C2 = run_plain(A, Bc, idx, m, n, k, N, M, V)
    assert bool(np.array_equal(C1.view(np.uint32), C2.view(np.uint32)))
    r = oracle.check(C1, oracle.spmm(A, Bc, idx, m, n, k, N, M, V), oracle.bound(A, Bc, idx, m, n, k, N, M, V))
    assert r, (name, r)


@pytest.mark.parametrize("shape", [(1, 8192, 8192, 4, 32, 64), (3, 4096, 11008, 8, 32, 32),
                                   (4, 2048, 8192, 16, 32, 32)], ids=lambda s: "x".join(map(str, s)))
def test_rowgather_default_dispatch(shape):
    """Decode batches of at most 4 rows take the row-gather kernel by default
    (no workspace, no split): every output within the bar, and the same
    result through the workspace entry point."""
    m, k, n, N, M, V = shape
    assert kname(m, n, k, N, M, V).startswith("nm_rowgather_kernel<r16,")
    assert ws_bytes(m, n, k, N, M, V) == 0
    C, C_ref, Bnd = parity(m, k, n, N, M, V, "normal", 61 + m)
    r = oracle.check(C, C_ref, Bnd)
    assert r, r


def test_rowgather_graph_replay():
    """The row-gather launch captured in a HIP graph (one kernel, nothing to
    clear first): every replay, with eager work between replays, gives the
    eager result bit for bit."""
    m, k, n, N, M, V = 2, 4096, 8192, 4, 32, 64
    name = kname(m, n, k, N, M, V)
    say(f"[graph] {name}")
    assert name.startswith("nm_rowgather_kernel<")
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 79, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    dA, dBc, didx = to_dev(A), to_dev(Bc), to_dev(idx)
    dC = torch.empty((m, n), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        nm.nmspmm_run(dA, dBc, didx, dC, m, n, k, N, M, V)
    torch.cuda.synchronize()
    eager = dC.cpu().numpy().copy()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        nm.nmspmm_run(dA, dBc, didx, dC, m, n, k, N, M, V)
    for i in range(3):
        dC.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert bool(np.array_equal(dC.cpu().numpy().view(np.uint32), eager.view(np.uint32))), f"replay {i}"


# every instantiated variant {RT, CT, NW, D}; tests/test_abi.py checks this list against the source
ROWGATHER_VARIANTS = [
    (1, 2, 8, 4), (1, 2, 8, 8), (1, 2, 16, 4), (1, 2, 16, 8),
    (1, 4, 8, 4), (1, 4, 8, 8), (1, 4, 16, 4), (1, 4, 16, 8),
    (2, 2, 8, 4), (2, 2, 16, 4), (2, 4, 8, 4), (2, 4, 16, 4),
]
# per row-tile count: a ragged shape (w = 291, quads spanning windows) with V a multiple of 64
ROWGATHER_VARIANT_SHAPES = {1: (13, 776, 512, 3, 8, 64), 2: (27, 776, 512, 3, 8, 64)}


@pytest.mark.parametrize("variant", ROWGATHER_VARIANTS, ids=lambda v: "rt%d_ct%d_nw%d_d%d" % v)
def test_rowgather_variants_exact(variant):
    """Every row-gather instantiation, forced: bit-exact on small integers and
    within the bar on normal data."""
    rt, ct, nw, d = variant
    for key, val in (("RG", 1), ("RGCT", ct), ("RGNW", nw), ("RGD", d)):
        TUNE[key] = str(val)
    m, k, n, N, M, V = ROWGATHER_VARIANT_SHAPES[rt]
    name = kname(m, n, k, N, M, V)
    say(f"[rowgather variant] {variant} {name}")
    assert name == f"nm_rowgather_kernel<r{16 * rt},c{16 * ct},w{nw},d{d}>,split1"
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 47 + m, "int")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C = run_plain(A, Bc, idx, m, n, k, N, M, V)
    assert bool(np.array_equal(C.astype(np.float64), oracle.spmm(A, Bc, idx, m, n, k, N, M, V)))
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 53 + m, "normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C = run_plain(A, Bc, idx, m, n, k, N, M, V)
    r = oracle.check(C, oracle.spmm(A, Bc, idx, m, n, k, N, M, V), oracle.bound(A, Bc, idx, m, n, k, N, M, V))
    assert r, (name, r)


# ---- device packer (nmspmm_compress_device) ----
PACK_SHAPES = [
    (64, 96, 4, 32, 32), (256, 256, 16, 32, 32), (128, 128, 8, 32, 64), (48, 30, 3, 8, 3),
    (28, 21, 2, 7, 3), (64, 64, 32, 32, 32), (64, 64, 1, 32, 16), (512, 256, 12, 32, 32),
    (512, 48, 5, 256, 16), (1024, 4096, 4, 32, 64),
    # LDS tile cut to 6 of 32 blocks (ragged last tile); per-thread packer (1024-wide blocks)
    (256, 512, 8, 128, 16), (64, 2048, 4, 32, 1024),
]


def device_pack(B, N, M, V):
    k, n = B.shape
    w = (k // M) * N
    dBc = torch.full((w, n), float("nan"), dtype=torch.float32, device="cuda")
    didx = torch.full((w, n // V), 255, dtype=torch.uint8, device="cuda")
    nm.nmspmm_compress_device(to_dev(B), dBc, didx, N, M, V)
    torch.cuda.synchronize()
    return dBc.cpu().numpy(), didx.cpu().numpy()


@pytest.mark.parametrize("kind", ["pruned", "dense", "ties", "zeros"])
@pytest.mark.parametrize("shape", PACK_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_compress_device_matches_oracle_byte_for_byte(shape, kind):
    k, n, N, M, V = shape
    if kind == "pruned":
        _, B, _ = make_inputs(1, k, n, N, M, V, seed=k + n, dist="normal")
    elif kind == "dense":
        B = np.random.default_rng(k * n).standard_normal((k, n)).astype(np.float32)
    elif kind == "ties":   # repeated row-vectors: every selection is decided by the tie rule
        B = np.repeat(np.random.default_rng(7).integers(-2, 3, (k // 2, n)), 2, axis=0).astype(np.float32)
    else:
        B = np.zeros((k, n), np.float32)
    Bc, idx = device_pack(B, N, M, V)
    Bc_o, idx_o = oracle.compress(B, N, M, V)
    assert np.array_equal(idx, idx_o)
    assert Bc.tobytes() == Bc_o.tobytes()


def test_device_pack_then_run_matches_host_pipeline():
    m, k, n, N, M, V = 512, 2048, 1024, 8, 32, 32
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 77)
    Bc, idx = device_pack(Bp, N, M, V)
    Bc_h, idx_h = nm.nmspmm_compress(Bp, N, M, V)
    assert np.array_equal(idx, idx_h) and Bc.tobytes() == Bc_h.tobytes()
    C = gpu_run(A, Bc, idx, m, n, k, N, M, V)
    r = oracle.check(C, oracle.spmm(A, Bc_h, idx_h, m, n, k, N, M, V), oracle.bound(A, Bc_h, idx_h, m, n, k, N, M, V))
    assert r, r
