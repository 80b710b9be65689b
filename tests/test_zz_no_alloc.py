"""nmspmm_run_noalloc (workspace in the library's static device scratch array,
for callers that cannot allocate) against nmspmm_run_ws with a caller-owned
workspace: the same kernels, so the outputs must be identical bit for bit,
on consecutive calls that share the array, each later call smaller than the
one before.  Both are also held to the oracle's bar (Eq. 1)."""
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

# (m, k, n, N, M, V), largest first: the direct-gather kernel at 128 rows
# (transposed A and offsets in the scratch), the pipelined streaming kernel
# with split-k partial tiles in the scratch (V = 16 keeps the gather kernel
# out), the direct-gather kernel at 40 rows, and the register-operand
# streaming kernel, which takes no scratch at all; then the direct-gather
# kernel in two row halves of 64 rows (128 rows on short strips).
CASES = [
    (128, 8192, 8192, 4, 32, 64),
    (64, 4096, 2048, 4, 32, 16),
    (40, 1536, 8192, 4, 32, 64),
    (16, 2048, 1024, 4, 32, 64),
    (128, 2048, 8192, 4, 32, 64),
]


def say(msg):
    print(msg, file=sys.stderr, flush=True)


def test_noalloc_matches_run_ws_on_consecutive_calls():
    names = []
    for m, k, n, N, M, V in CASES:
        need = nm.nmspmm_workspace_bytes(m, n, k, N, M, V)
        name = nm.nmspmm_kernel_name_ws(m, n, k, N, M, V)
        names.append(name)
        say(f"[noalloc] m={m} k={k} n={n} {N}:{M} V={V} {name} workspace={need}")
        assert need <= nm.NMSPMM_NOALLOC_SCRATCH_BYTES
        A, Bp, _ = make_inputs(m, k, n, N, M, V, 500 + m, "normal")
        Bc, idx = nm.nmspmm_compress(Bp, N, M, V)
        dA, dBc, didx = (torch.from_numpy(x).cuda() for x in (A, Bc, idx))
        ws = torch.full((max(need, 1),), 0xFF, dtype=torch.uint8, device="cuda")
        ref = torch.full((m, n), float("nan"), device="cuda")
        nm.nmspmm_run_ws(dA, dBc, didx, ref, m, n, k, N, M, V, ws if need > 0 else None)
        out = torch.full((m, n), float("nan"), device="cuda")
        nm.nmspmm_run_noalloc(dA, dBc, didx, out, m, n, k, N, M, V)
        torch.cuda.synchronize()
        C_ws, C_na = ref.cpu().numpy(), out.cpu().numpy()
        C_ref = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
        Bnd = oracle.bound(A, Bc, idx, m, n, k, N, M, V)
        if "+zero,split" in name and not name.endswith("split1"):
            # no scratch: split-k adds with fp32 atomics, whose order (and so
            # the last bits) varies between runs; both meet the bar
            assert oracle.check(C_ws, C_ref, Bnd)
        else:
            assert bool(np.array_equal(C_ws.view(np.uint32), C_na.view(np.uint32))), \
                f"{name}: {int(np.count_nonzero(C_ws != C_na))} outputs differ"
        r = oracle.check(C_na, C_ref, Bnd)
        say(f"[noalloc] {name}: {r}")
        assert r, (name, r)
    assert names[0].startswith("nm_gather_kernel<r128,") and "+ws,split" in names[1]
    assert names[2].startswith("nm_gather_kernel<r64,") and names[3].startswith("nm_skinny_kernel")
    assert names[4].startswith("nm_gather_kernel<r64x2,")


def test_noalloc_epilogue_matches_run_ws():
    """The fused epilogue (alpha = M/N, bias, GELU) through the static scratch."""
    m, k, n, N, M, V = 64, 4096, 2048, 4, 32, 64
    A, Bp, _ = make_inputs(m, k, n, N, M, V, 901, "normal")
    Bc, idx = nm.nmspmm_compress(Bp, N, M, V)
    dA, dBc, didx = (torch.from_numpy(x).cuda() for x in (A, Bc, idx))
    bias = torch.randn(n, device="cuda")
    ws = torch.empty(nm.nmspmm_workspace_bytes(m, n, k, N, M, V), dtype=torch.uint8, device="cuda")
    ref = torch.empty((m, n), device="cuda")
    out = torch.full((m, n), float("nan"), device="cuda")
    nm.nmspmm_run_ws(dA, dBc, didx, ref, m, n, k, N, M, V, ws, alpha=M / N, bias=bias, act="gelu")
    nm.nmspmm_run_noalloc(dA, dBc, didx, out, m, n, k, N, M, V, alpha=M / N, bias=bias, act="gelu")
    torch.cuda.synchronize()
    assert torch.equal(ref.view(torch.int32), out.view(torch.int32))
