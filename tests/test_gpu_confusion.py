"""GPU parity of Eq. 2's confusion matrix (Sec. II-A),
W[i][j] = |C'[i][j] - C[i][j]| / (m*n), through the C ABI against the CPU
oracle.

- nmspmm_confusion alone: every output is the fp64 quotient rounded once to
  fp32, so it must equal the oracle's fp64 W rounded to fp32 bit for bit.
- The whole diagnostic on the GPU: C' = nmspmm_run_ex with alpha = M/N on
  the device packer's (Bc, idx) of an unpruned B, C = nmspmm_run on the
  N = M packing of the same B (every row kept: the dense product), then W.
  Each product is within 1e-5 * sum |A||B| of its fp64 reference, so W is
  within 1e-5 * ((M/N) * Bnd' + Bnd) / (m*n) of the oracle's, plus the
  rounding of W itself.
"""
import sys

import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2503_01253_amd as nm  # noqa: E402


def say(msg):
    print(msg, file=sys.stderr, flush=True)


def to_dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


@pytest.mark.parametrize("m,n", [(1, 1), (1, 3), (3, 5), (4, 4), (257, 129), (1024, 1000), (2048, 4096)])
@pytest.mark.parametrize("offset", [0, 1])
def test_confusion_kernel_bit_exact(m, n, offset):
    """offset 1 starts every array one float past a 16-byte boundary: the
    kernel's 4-byte path; offset 0 takes the 16-byte path and its tail."""
    say(f"[confusion] kernel m={m} n={n} offset={offset}")
    rng = np.random.default_rng(m * 7 + n + offset)
    Cs = rng.standard_normal((m, n)).astype(np.float32)
    Cd = (Cs + rng.standard_normal((m, n)).astype(np.float32) * 1e-3).astype(np.float32)
    Cd[0, 0] = Cs[0, 0]   # one exact zero
    ref = oracle.confusion(Cs.astype(np.float64), Cd.astype(np.float64)).astype(np.float32)
    bufs = [torch.full((m * n + offset,), float("nan"), dtype=torch.float32, device="cuda") for _ in range(3)]
    dS, dD, dW = (b[offset:].view(m, n) for b in bufs)
    dS.copy_(to_dev(Cs))
    dD.copy_(to_dev(Cd))
    st = nm.lib().nmspmm_confusion(dS.data_ptr(), dD.data_ptr(), dW.data_ptr(), m, n,
                                   torch.cuda.current_stream().cuda_stream)
    assert st == nm.NMSPMM_OK
    torch.cuda.synchronize()
    W = dW.cpu().numpy()
    assert np.array_equal(W, ref)
    assert W[0, 0] == 0.0
    # in place, over the sparse output
    nm.nmspmm_confusion(dS, dD, dS)
    torch.cuda.synchronize()
    assert np.array_equal(dS.cpu().numpy(), ref)
    # the floats around the arrays are untouched
    if offset:
        assert torch.isnan(bufs[2][0]).item()


def test_confusion_special_values():
    """Infinities and NaN propagate as the fp64 formula says; the result is
    never negative."""
    Cs = np.array([[np.inf, 1.0, -2.0, np.nan, 0.0, -0.0, 3e38, -3e38]], np.float32)
    Cd = np.array([[1.0, np.inf, -2.0, 1.0, -0.0, 0.0, -3e38, 3e38]], np.float32)
    ref = oracle.confusion(Cs.astype(np.float64), Cd.astype(np.float64)).astype(np.float32)
    dW = torch.empty((1, 8), dtype=torch.float32, device="cuda")
    nm.nmspmm_confusion(to_dev(Cs), to_dev(Cd), dW)
    torch.cuda.synchronize()
    W = dW.cpu().numpy()
    np.testing.assert_array_equal(W, ref)
    assert not np.signbit(W[0, 4]) and not np.signbit(W[0, 5])


CHAIN = [
    (300, 320, 320, 16, 32, 32),
    (1030, 128, 1088, 4, 32, 32),
    (130, 1024, 2048, 4, 32, 64),
    (64, 256, 512, 8, 32, 32),
    (17, 24, 10, 3, 8, 2),
    (16, 8192, 8192, 4, 32, 64),
    (4096, 4096, 4096, 16, 32, 32),
]


@pytest.mark.parametrize("shape", CHAIN, ids=lambda s: "x".join(map(str, s)))
def test_eq2_diagnostic_chain(shape):
    m, k, n, N, M, V = shape
    say(f"[confusion] chain m={m} k={k} n={n} {N}:{M} V={V}")
    rng = np.random.default_rng(m + 3 * k + 5 * n)
    A = rng.uniform(-1, 1, (m, k)).astype(np.float32)
    B = rng.uniform(-1, 1, (k, n)).astype(np.float32)      # unpruned
    dA, dB = to_dev(A), to_dev(B)
    w = (k // M) * N
    dBc = torch.empty((w, n), dtype=torch.float32, device="cuda")
    didx = torch.empty((w, n // V), dtype=torch.uint8, device="cuda")
    nm.nmspmm_compress_device(dB, dBc, didx, N, M, V)
    dBd = torch.empty((k, n), dtype=torch.float32, device="cuda")
    didd = torch.empty((k, n // V), dtype=torch.uint8, device="cuda")
    nm.nmspmm_compress_device(dB, dBd, didd, M, M, V)
    dCs = torch.empty((m, n), dtype=torch.float32, device="cuda")
    dCd = torch.empty((m, n), dtype=torch.float32, device="cuda")
    alpha = M / N
    nm.nmspmm_run_ex(dA, dBc, didx, dCs, m, n, k, N, M, V, alpha=alpha)
    nm.nmspmm_run(dA, dBd, didd, dCd, m, n, k, M, M, V)
    dW = torch.full((m, n), float("nan"), dtype=torch.float32, device="cuda")
    nm.nmspmm_confusion(dCs, dCd, dW)
    torch.cuda.synchronize()
    W = dW.cpu().numpy().astype(np.float64)

    Bc, idx = oracle.compress(B, N, M, V)
    assert np.array_equal(didx.cpu().numpy(), idx) and np.array_equal(dBc.cpu().numpy(), Bc)
    Cs_ref = oracle.epilogue(oracle.spmm(A, Bc, idx, m, n, k, N, M, V), alpha=alpha)
    Cd_ref = oracle.dense(A, B)
    W_ref = oracle.confusion(Cs_ref, Cd_ref)
    Bd, idd = oracle.compress(B, M, M, V)
    bnd = (alpha * oracle.bound(A, Bc, idx, m, n, k, N, M, V) * (1 + 1e-6)
           + oracle.bound(A, Bd, idd, m, n, k, M, M, V)) / (m * n)
    tol = oracle.PARITY_RTOL * bnd + 2.0 ** -23 * np.abs(W_ref)
    assert np.all(np.isfinite(W)) and np.all(W >= 0)
    err = np.abs(W - W_ref)
    assert np.all(err <= tol), f"worst err/tol {float(np.max(err / tol)):.3f}"
    # the diagnostic's one-number summary: the mean absolute error of C'
    mae, mae_ref = W.sum(), W_ref.sum()
    assert abs(mae - mae_ref) <= tol.sum() + 1e-6 * mae_ref
