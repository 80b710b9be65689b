"""Pins for the CPU oracle: checks against what the mathematics fixes, never
against the oracle itself (Sec. II-A, Eq. 1 as read in the oracle's header)."""
import json
import os

import numpy as np
import pytest

import oracle
from nm_workloads import make_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

# (m, k, n, N, M, V): tiny shapes over a spread of N:M and vector lengths
TINY = [
    (5, 8, 12, 1, 4, 1),
    (7, 16, 16, 2, 4, 4),
    (3, 24, 10, 3, 8, 2),
    (9, 64, 64, 16, 32, 32),
    (4, 64, 32, 32, 32, 8),
    (6, 35, 9, 5, 7, 3),
    (1, 32, 64, 4, 32, 64),
    (8, 64, 40, 8, 32, 8),
]


def dense_sequential(A, B):
    """Dense product in fp64, adding the k terms in increasing k for every
    output (a textbook GEMM with a fixed summation order)."""
    A64 = A.astype(np.float64)
    B64 = B.astype(np.float64)
    C = np.zeros((A.shape[0], B.shape[1]), dtype=np.float64)
    for kk in range(A.shape[1]):
        C += np.outer(A64[:, kk], B64[kk, :])
    return C


@pytest.mark.parametrize("shape", TINY)
@pytest.mark.parametrize("dist", ["uniform", "normal"])
def test_brute_force_bit_exact(shape, dist):
    """oracle_spmm on (Bc, idx) == dense fp64 product on the pruned B, bit for bit.
    Pruned terms contribute exact zeros, fp32 products are exact in fp64 and
    the kept rows are visited in increasing k on both sides."""
    m, k, n, N, M, V = shape
    A, Bp, _ = make_inputs(m, k, n, N, M, V, seed=11 + m * k + n, dist=dist)
    Bc, idx = oracle.compress(Bp, N, M, V)
    C = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    assert np.array_equal(C, dense_sequential(A, Bp))


@pytest.mark.parametrize("M,V", [(4, 1), (8, 4), (32, 32), (32, 64)])
def test_dense_case_N_equals_M(M, V):
    """0% sparsity (N = M, Sec. IV-B) is a plain dense GEMM: every offset is
    kept in order and Bc is B itself."""
    m, k, n = 6, 2 * M, 2 * V
    rng = np.random.default_rng(5)
    A = rng.uniform(-1, 1, (m, k)).astype(np.float32)
    B = rng.uniform(-1, 1, (k, n)).astype(np.float32)
    Bc, idx = oracle.compress(B, M, M, V)
    assert np.array_equal(Bc, B)
    u = np.arange(k)
    assert np.array_equal(idx, np.repeat((u % M)[:, None], n // V, axis=1))
    C = oracle.spmm(A, Bc, idx, m, n, k, M, M, V)
    ref = A.astype(np.float64) @ B.astype(np.float64)  # library GEMM, its own order
    assert np.allclose(C, ref, rtol=0, atol=1e-12 * np.abs(A).sum())


@pytest.mark.parametrize("N,M,V", [(2, 4, 4), (3, 8, 2), (16, 32, 32)])
def test_identity_returns_pruned_B(N, M, V):
    k = 2 * M
    n = 3 * V
    _, Bp, _ = make_inputs(1, k, n, N, M, V, seed=3)
    Bc, idx = oracle.compress(Bp, N, M, V)
    C = oracle.spmm(np.eye(k, dtype=np.float32), Bc, idx, k, n, k, N, M, V)
    assert np.array_equal(C, Bp.astype(np.float64))


@pytest.mark.parametrize("N,M,n", [(2, 4, 12), (3, 8, 7), (4, 32, 64), (16, 32, 40)])
def test_one_block_is_column_gather_then_dense_gemm(N, M, n):
    """V = n (one column block, Sec. II-A): every column of C uses the same
    kept k-rows, so C is A restricted to the kept columns times B restricted
    to the kept rows.  The kept set comes from the generator's mask, not from
    idx, and the product is a library GEMM (its own order, so to fp64
    rounding) and a sequential-k dense sum (bit for bit)."""
    m, k = 5, 4 * M
    A, Bp, mask = make_inputs(m, k, n, N, M, n, seed=31 + N + M, dist="normal")
    kept = np.nonzero(mask[:, 0])[0]
    assert len(kept) == (k // M) * N and np.all(mask == mask[:, :1])
    Bc, idx = oracle.compress(Bp, N, M, n)
    assert np.array_equal(Bc, Bp[kept])                  # compressed rows = kept rows, in k order
    C = oracle.spmm(A, Bc, idx, m, n, k, N, M, n)
    Ag = np.ascontiguousarray(A[:, kept])
    assert np.array_equal(C, dense_sequential(Ag, Bp[kept]))
    ref = Ag.astype(np.float64) @ Bp[kept].astype(np.float64)
    scale = np.abs(Ag.astype(np.float64)) @ np.abs(Bp[kept].astype(np.float64))
    assert np.all(np.abs(C - ref) <= 1e-14 * scale)


@pytest.mark.parametrize("N,M,V,k,n", [(2, 4, 4, 48, 16), (3, 8, 2, 48, 6), (1, 4, 1, 52, 5),
                                       (4, 16, 8, 48, 24)])
def test_bitmask_encoding(N, M, V, k, n):
    """With A[0][kk] = 2^kk and every kept value 1, each output is the integer
    whose set bits are exactly the k-rows its column block kept: this pins the
    window base floor(u/N)*M, the offset lookup by column block and the
    absence of any rescaling, independently of the oracle's own loops."""
    _, _, mask = make_inputs(1, k, n, N, M, V, seed=21)
    Bp = mask.astype(np.float32)
    A = np.zeros((2, k), dtype=np.float32)
    A[0] = 2.0 ** np.arange(k)
    A[1] = 1.0
    Bc, idx = oracle.compress(Bp, N, M, V)
    C = oracle.spmm(A, Bc, idx, 2, n, k, N, M, V)
    for j in range(n):
        expect = sum(1 << kk for kk in range(k) if mask[kk, j])
        assert int(C[0, j]) == expect and C[0, j] == float(expect)
    assert np.all(C[1] == (k // M) * N)


def test_hand_example_fig1_parameters():
    g = json.load(open(os.path.join(GOLDEN, "fig1_hand_example.json")))
    N, M, V, m, k, n = g["N"], g["M"], g["V"], g["m"], g["k"], g["n"]
    idx = np.array(g["idx"], dtype=np.uint8)
    A = np.array(g["A"], dtype=np.float32)
    Bc = np.full(((k // M) * N, n), g["Bc_value"], dtype=np.float32)
    C = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    assert np.array_equal(C, np.array(g["C_expected"], dtype=np.float64))
    # the compressor rebuilds the same idx from the dense pattern
    Bd = np.zeros((k, n), dtype=np.float32)
    for key, rows in g["kept_rows"].items():
        if key == "comment":
            continue
        b = int(key.split("_b")[1])
        for r in rows:
            Bd[r, b * V:(b + 1) * V] = 1.0
    Bc2, idx2 = oracle.compress(Bd, N, M, V)
    assert np.array_equal(idx2, idx)
    assert np.array_equal(Bc2, Bc)


@pytest.mark.parametrize("shape", TINY)
def test_compress_invariants_and_round_trip(shape):
    m, k, n, N, M, V = shape
    _, Bp, mask = make_inputs(m, k, n, N, M, V, seed=77)
    Bc, idx = oracle.compress(Bp, N, M, V)
    w, q = (k // M) * N, n // V
    assert Bc.shape == (w, n) and idx.shape == (w, q)
    assert oracle.validate(idx, k, n, N, M, V) == 0
    # exactly N strictly increasing offsets < M per (group, block)
    d = idx.reshape(k // M, N, q).astype(int)
    assert np.all(d < M)
    if N > 1:
        assert np.all(np.diff(d, axis=1) > 0)
    # the kept set is the generator's mask, and the values round-trip
    rec = np.zeros((k, q), dtype=bool)
    for u in range(w):
        for b in range(q):
            rec[(u // N) * M + idx[u, b], b] = True
    assert np.array_equal(np.repeat(rec, V, axis=1), mask)
    assert np.array_equal(oracle.decompress(Bc, idx, k, n, N, M, V), Bp)
    # Bc rows are the kept source vectors
    for u in range(w):
        for b in range(q):
            r = (u // N) * M + idx[u, b]
            assert np.array_equal(Bc[u, b * V:(b + 1) * V], Bp[r, b * V:(b + 1) * V])


def test_compress_selection_rule_on_dense_input():
    """On an unpruned B the kept rows are the N of largest squared norm over
    the block; no dropped row beats a kept one."""
    k, n, N, M, V = 64, 48, 3, 8, 4
    rng = np.random.default_rng(9)
    B = rng.standard_normal((k, n)).astype(np.float32)
    Bc, idx = oracle.compress(B, N, M, V)
    for g in range(k // M):
        for b in range(n // V):
            blk = B[g * M:(g + 1) * M, b * V:(b + 1) * V].astype(np.float64)
            s = (blk * blk).sum(axis=1)
            kept = set(int(o) for o in idx[g * N:(g + 1) * N, b])
            dropped = set(range(M)) - kept
            assert min(s[o] for o in kept) >= max(s[o] for o in dropped)


def test_compress_ties_go_to_smaller_offset():
    k, n, N, M, V = 8, 4, 2, 4, 2
    B = np.ones((k, n), dtype=np.float32)
    Bc, idx = oracle.compress(B, N, M, V)
    assert np.array_equal(idx, np.array([[0, 0], [1, 1], [0, 0], [1, 1]], dtype=np.uint8))


def test_validate_flags_bad_indices():
    k, n, N, M, V = 16, 8, 2, 8, 4
    _, Bp, _ = make_inputs(1, k, n, N, M, V, seed=1)
    _, idx = oracle.compress(Bp, N, M, V)
    assert oracle.validate(idx, k, n, N, M, V) == 0
    bad = idx.copy()
    bad[0, 0] = M
    assert oracle.validate(bad, k, n, N, M, V) == 2
    bad = idx.copy()
    bad[1, 0] = bad[0, 0]
    assert oracle.validate(bad, k, n, N, M, V) == 3
    assert oracle.validate(idx, k + 1, n, N, M, V) == 1


@pytest.mark.parametrize("shape", TINY[:5])
def test_bound_matches_library_matmul(shape):
    m, k, n, N, M, V = shape
    A, Bp, _ = make_inputs(m, k, n, N, M, V, seed=5, dist="normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    Bnd = oracle.bound(A, Bc, idx, m, n, k, N, M, V)
    ref = np.abs(A.astype(np.float64)) @ np.abs(Bp.astype(np.float64))
    assert np.allclose(Bnd, ref, rtol=1e-13, atol=0)


def test_matches_scipy_sparse_product():
    """A library sparse-matrix product on the pruned B agrees to fp64 rounding."""
    sp = pytest.importorskip("scipy.sparse")
    m, k, n, N, M, V = 33, 128, 96, 4, 32, 32
    A, Bp, _ = make_inputs(m, k, n, N, M, V, seed=123, dist="normal")
    Bc, idx = oracle.compress(Bp, N, M, V)
    C = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    Bnd = oracle.bound(A, Bc, idx, m, n, k, N, M, V)
    ref = np.asarray((sp.csr_matrix(Bp.astype(np.float64)).T @ A.astype(np.float64).T).T)
    assert np.all(np.abs(C - ref) <= 1e-14 * Bnd + 1e-300)


def test_degenerate_shapes():
    # k = 0: no terms, C = 0
    C = oracle.spmm(np.zeros((3, 0), np.float32), np.zeros((0, 8), np.float32),
                    np.zeros((0, 2), np.uint8), 3, 8, 0, 2, 4, 4)
    assert C.shape == (3, 8) and np.all(C == 0)
    # m = 0: empty output
    C = oracle.spmm(np.zeros((0, 8), np.float32), np.zeros((4, 8), np.float32),
                    np.zeros((4, 2), np.uint8), 0, 8, 8, 2, 4, 4)
    assert C.shape == (0, 8)
    with pytest.raises(ValueError):
        oracle.compress(np.zeros((9, 8), np.float32), 2, 4, 4)   # k % M != 0
    with pytest.raises(ValueError):
        oracle.compress(np.zeros((8, 6), np.float32), 2, 4, 4)   # n % V != 0
    with pytest.raises(ValueError):
        oracle.compress(np.zeros((8, 8), np.float32), 5, 4, 4)   # N > M


def test_checker_rejects_injected_errors():
    m, k, n, N, M, V = 8, 64, 64, 8, 32, 32
    A, Bp, _ = make_inputs(m, k, n, N, M, V, seed=2)
    Bc, idx = oracle.compress(Bp, N, M, V)
    C = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    Bnd = oracle.bound(A, Bc, idx, m, n, k, N, M, V)
    assert oracle.check(C.astype(np.float32), C, Bnd)
    bad = C.copy()
    bad[3, 7] += 2 * oracle.PARITY_RTOL * Bnd[3, 7]
    r = oracle.check(bad, C, Bnd)
    assert not r and r.n_bad == 1 and tuple(r.worst_index) == (3, 7)
    bad = C.copy()
    bad[0, 0] = np.nan
    r = oracle.check(bad, C, Bnd)
    assert not r and r.n_nonfinite == 1
    bad = C.copy()
    bad[1, 1] = np.inf
    assert not oracle.check(bad, C, Bnd)
    # a dropped term (one kept row missing) is far outside the tolerance
    Bc2 = Bc.copy()
    Bc2[5] = 0
    C2 = oracle.spmm(A, Bc2, idx, m, n, k, N, M, V)
    assert not oracle.check(C2, C, Bnd)


def test_epilogue_pins():
    """alpha, bias and activation against closed forms and scipy's normal CDF
    (an independent implementation of Phi)."""
    from scipy.stats import norm
    rng = np.random.default_rng(5)
    C = rng.standard_normal((7, 9)) * 3
    bias = rng.standard_normal(9).astype(np.float32)
    np.testing.assert_array_equal(oracle.epilogue(C), C)
    np.testing.assert_array_equal(oracle.epilogue(C, alpha=4.0), 4.0 * C)   # Eq. 1's M/N at 8:32
    np.testing.assert_array_equal(oracle.epilogue(C, bias=bias), C + bias.astype(np.float64))
    np.testing.assert_array_equal(oracle.epilogue(C, act="relu"), np.maximum(C, 0.0))
    y = 2.0 * C + bias.astype(np.float64)
    np.testing.assert_allclose(oracle.epilogue(C, 2.0, bias, "gelu"), y * norm.cdf(y), rtol=1e-13, atol=1e-15)
    g = oracle.epilogue(np.array([[0.0, 40.0, -40.0, 1.0]]), act="gelu")
    assert g[0, 0] == 0.0 and g[0, 1] == 40.0 and g[0, 2] == 0.0
    assert abs(g[0, 3] - 0.8413447460685429) < 1e-15          # Phi(1)
    with pytest.raises(ValueError):
        oracle.epilogue(C, bias=np.zeros(3, np.float32))


def test_eq2_hand_example():
    """Eq. 2 on a hand-worked case: selection, Eq. 1 with its M/N factor,
    the dense product and W, every value written out by hand."""
    g = json.load(open(os.path.join(GOLDEN, "eq2_hand_example.json")))
    N, M, V, m, k, n = g["N"], g["M"], g["V"], g["m"], g["k"], g["n"]
    A = np.array(g["A"], np.float32)
    B = np.array(g["B"], np.float32)
    Bc, idx = oracle.compress(B, N, M, V)
    assert np.array_equal(idx, np.array(g["idx"], np.uint8))
    assert np.array_equal(Bc, np.array(g["Bc"], np.float32))
    Cu = oracle.spmm(A, Bc, idx, m, n, k, N, M, V)
    assert np.array_equal(Cu, np.array(g["C_sparse_unscaled"], np.float64))
    Cs = oracle.epilogue(Cu, alpha=M / N)
    assert np.array_equal(Cs, np.array(g["C_sparse"], np.float64))
    C = oracle.dense(A, B)
    assert np.array_equal(C, np.array(g["C_dense"], np.float64))
    W = oracle.confusion(Cs, C)
    assert np.array_equal(W, np.array(g["W_expected"], np.float64))


@pytest.mark.parametrize("shape", TINY)
def test_dense_matches_sequential_product_and_spmm_at_N_equals_M(shape):
    """oracle_dense is the textbook product: bit for bit the sequential-k
    fp64 sum, and bit for bit oracle_spmm on the N = M compression (every row
    kept, the same order of additions)."""
    m, k, n, _, M, V = shape
    rng = np.random.default_rng(k * n + m)
    A = rng.uniform(-1, 1, (m, k)).astype(np.float32)
    B = rng.uniform(-1, 1, (k, n)).astype(np.float32)
    C = oracle.dense(A, B)
    assert np.array_equal(C, dense_sequential(A, B))
    Bc, idx = oracle.compress(B, M, M, V)
    assert np.array_equal(C, oracle.spmm(A, Bc, idx, m, n, k, M, M, V))
    ref = A.astype(np.float64) @ B.astype(np.float64)   # library GEMM, its own order
    assert np.allclose(C, ref, rtol=0, atol=1e-12 * np.abs(A).sum())


@pytest.mark.parametrize("shape", TINY)
def test_confusion_closed_form_on_pruned_B(shape):
    """When B is already pruned, C = A*Bp and C' = (M/N)*A*Bp, so Eq. 2 has
    the closed form W = (M/N - 1) * |A*Bp| / (m*n); at N = M it is zero."""
    m, k, n, N, M, V = shape
    A, Bp, _ = make_inputs(m, k, n, N, M, V, seed=41 + m + k)
    Bc, idx = oracle.compress(Bp, N, M, V)
    Cs = oracle.epilogue(oracle.spmm(A, Bc, idx, m, n, k, N, M, V), alpha=M / N)
    W = oracle.confusion(Cs, oracle.dense(A, Bp))
    AB = A.astype(np.float64) @ Bp.astype(np.float64)
    ref = (M / N - 1.0) * np.abs(AB) / (m * n)
    scale = (M / N + 1.0) * (np.abs(A).astype(np.float64) @ np.abs(Bp).astype(np.float64)) / (m * n)
    assert np.all(np.abs(W - ref) <= 1e-12 * scale)
    if N == M:
        assert np.array_equal(W, np.zeros_like(W))


def test_confusion_elementwise_properties():
    """W is |difference| / (m*n): symmetric in its two arguments, zero on
    equal inputs, and linear in a power-of-two scale (exact in binary)."""
    rng = np.random.default_rng(3)
    a = rng.standard_normal((5, 6))
    b = rng.standard_normal((5, 6))
    W = oracle.confusion(a, b)
    assert np.array_equal(W, oracle.confusion(b, a))
    assert np.array_equal(oracle.confusion(a, a), np.zeros_like(a))
    assert np.array_equal(oracle.confusion(8 * a, 8 * b), 8 * W)
    assert np.array_equal(oracle.confusion(np.array([[3.0]]), np.array([[-1.0]])), np.array([[4.0]]))
    with pytest.raises(ValueError):
        oracle.confusion(a, b[:, :5])
