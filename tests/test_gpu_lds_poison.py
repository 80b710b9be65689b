"""Race detection for the LDS pipelines: every kernel family that fills LDS by
buffer->LDS DMA (the tiled kernel's Bc and offset stages and its A_s slots,
the pipelined streaming kernel's ring, the register-operand streaming
kernel's A chunks) run from the library's debug twin, built with
NMSPMM_POISON_LDS=1.  There every LDS fill first writes NaN (or, for offset
bytes, an out-of-window value that the readers clamp to a wrong column) into
its destination, so a read that runs ahead of a wait or a barrier sees
poison instead of stale data that may happen to be right.  With small-integer
inputs every correct result is exact, so any such read fails the comparison.
The variants are forced through the tuning entry point, on ragged shapes with
partial stages and split-k."""
import ctypes
import sys

import numpy as np
import pytest

import oracle
from nm_workloads import make_inputs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2503_01253_amd as nm  # noqa: E402
from paper_2503_01253_amd.binding import load, tuning_string  # noqa: E402
from paper_2503_01253_amd.build import POISON_LIB_PATH  # noqa: E402

L = load(POISON_LIB_PATH)


def say(msg):
    print(msg, file=sys.stderr, flush=True)


def variant_name(shape, tune):
    m, k, n, N, M, V = shape
    return L.nmspmm_kernel_name_tuned(m, n, k, N, M, V, 0, tuning_string(tune)).decode()


def poisoned_run(shape, tune, seed):
    """Name of the forced variant, and the number of outputs that differ from
    the oracle (exact on small integers) when it runs from the poisoned
    library."""
    m, k, n, N, M, V = shape
    ts = tuning_string(tune)
    name = variant_name(shape, tune)
    A, Bp, _ = make_inputs(m, k, n, N, M, V, seed, "int")
    Bc, idx = oracle.compress(Bp, N, M, V)
    dA, dBc, didx = (torch.from_numpy(x).cuda() for x in (A, Bc, idx))
    dC = torch.full((m, n), float("nan"), device="cuda")
    say(f"[poison] {shape} {tune} {name}")
    st = L.nmspmm_run_tuned(dA.data_ptr(), dBc.data_ptr(), didx.data_ptr(), dC.data_ptr(), m, n, k, N, M, V,
                            ctypes.c_float(1.0), None, 0, None, 0, ts, torch.cuda.current_stream().cuda_stream)
    assert st == 0, nm.nmspmm_status_string(st)
    torch.cuda.synchronize()
    C = dC.cpu().numpy().astype(np.float64)
    C_ref = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    bad = int(np.count_nonzero(C != C_ref))
    return name, bad


TILES = ["256x256", "128x512", "128x128", "64x512", "16x512", "128x256", "256x128", "256x256m32", "128x512m32",
         "128x128m32", "64x512m32", "128x256m32", "64x1024m32", "256x256m32w16", "128x512m32w16", "128x256m32w16"]
TILED_SHAPES = [
    (300, 256, 1088, 8, 32, 32),     # 8 windows, ragged m and n
    (130, 416, 1024, 4, 32, 64),     # 13 windows: a partial last stage at KA = 64 / 128
    (300, 288, 1088, 16, 32, 32),    # 16:32: the 16-wave tiles' stages of 32 rows at KA = 64, a partial last one
    (130, 192, 1024, 32, 32, 64),    # N = M: stages of 32 rows at KA = 32
]


@pytest.mark.parametrize("ka", [0, 64, 128])
@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("shape", TILED_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_tiled_kernel_under_poison(shape, tile, ka):
    tune = {"TILE": tile, "SPLITS": 2}
    if ka:
        tune["KA"] = ka
    name = variant_name(shape, tune)
    if f"<{tile}," not in name or (ka and f",ka{ka}," not in name):
        pytest.skip(f"not instantiated for {shape}: {name}")
    name, bad = poisoned_run(shape, tune, seed=3 + ka)
    assert bad == 0, f"{name}: {bad} outputs differ"


STREAM_SHAPES = [(70, 1000, 832, 3, 8, 64), (40, 1536, 512, 4, 32, 64)]
STREAM_VARIANTS = [(1, 1, 1, 16), (1, 2, 1, 32), (2, 2, 1, 16), (2, 1, 1, 32), (4, 1, 1, 16), (2, 2, 2, 16)]


@pytest.mark.parametrize("splits", [1, 3])
@pytest.mark.parametrize("variant", STREAM_VARIANTS, ids=lambda v: "rt%d_bv%d_cpw%d_rb%d" % v)
@pytest.mark.parametrize("shape", STREAM_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_stream_kernel_under_poison(shape, variant, splits):
    rt, bv, cpw, rb = variant
    tune = {"PS": 1, "PSRT": rt, "PSBV": bv, "PSCPW": cpw, "PSRB": rb, "SPLITS": splits, "GATHER": 0}
    name = variant_name(shape, tune)
    if not name.startswith("nm_stream_kernel<r%d,c%d,bv%d,rb%d>" % (16 * rt, 128 * bv * cpw, bv, rb)):
        pytest.skip(f"not available for {shape}: {name}")
    name, bad = poisoned_run(shape, tune, seed=5 + rt + rb)
    assert bad == 0, f"{name}: {bad} outputs differ"


SKINNY_SHAPES = [(16, 2048, 640, 4, 32, 64), (40, 1536, 256, 8, 32, 32)]


@pytest.mark.parametrize("splits", [1, 3])
@pytest.mark.parametrize("rt,cols,qpw", [(1, 128, 2), (1, 64, 4), (1, 256, 1), (2, 128, 2), (2, 256, 1)])
@pytest.mark.parametrize("shape", SKINNY_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_skinny_kernel_under_poison(shape, rt, cols, qpw, splits):
    tune = {"TILE": "skinny", "PS": 0, "RT": rt, "SKCOLS": cols, "QPW": qpw, "SPLITS": splits}
    name = variant_name(shape, tune)
    if not name.startswith(f"nm_skinny_kernel<c{cols},") or f"qpw{qpw}" not in name:
        pytest.skip(f"not instantiated for {shape}: {name}")
    name, bad = poisoned_run(shape, tune, seed=9 + cols)
    assert bad == 0, f"{name}: {bad} outputs differ"


def test_poisoned_library_is_a_separate_build():
    """The debug twin is another file than the product library, and the
    product library's dispatch names the same variants."""
    assert POISON_LIB_PATH != nm.binding.LIB_PATH
    shape = (4096, 4096, 4096, 16, 32, 32)
    assert L.nmspmm_kernel_name(*shape).decode() == nm.nmspmm_kernel_name(*shape)
