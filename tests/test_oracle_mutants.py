"""Pin strength: plant plausible mistakes in a copy of the oracle's C source
(on the CPU, in a temporary directory), rebuild it, and check that at least
one pin fails for every mistake.  The committed oracle is never modified."""
import ctypes
import json
import os

import numpy as np
import pytest

import oracle
from oracle.build import SRC, build
from nm_workloads import make_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

MUTANTS = {
    # Eq. 1 taken literally: window base u*M/N instead of floor(u/N)*M
    "literal_window": ("const int64_t window = (u / N) * M;\n            const float *brow",
                       "const int64_t window = u * M / N;\n            const float *brow"),
    # one compressed row dropped
    "dropped_term": ("for (int64_t u = 0; u < w; ++u) {\n            const int64_t window = (u / N) * M;\n            const float *brow = Bc + u * n;\n            const uint8_t *drow = idx + u * q;\n            for (int64_t b = 0; b < q; ++b) {\n                const double av = (double)",
                     "for (int64_t u = 0; u + 1 < w; ++u) {\n            const int64_t window = (u / N) * M;\n            const float *brow = Bc + u * n;\n            const uint8_t *drow = idx + u * q;\n            for (int64_t b = 0; b < q; ++b) {\n                const double av = (double)"),
    # offsets looked up in the wrong column block
    "wrong_block": ("const double av = (double)a[window + drow[b]];",
                    "const double av = (double)a[window + drow[q - 1 - b]];"),
    # Eq. 1's M/N factor applied
    "scaled": ("for (int64_t jj = 0; jj < V; ++jj) cb[jj] += av * (double)bb[jj];\n            }\n        }\n    }\n    return 0;\n}\n\n/* The magnitude",
               "for (int64_t jj = 0; jj < V; ++jj) cb[jj] += (double)M / N * av * (double)bb[jj];\n            }\n        }\n    }\n    return 0;\n}\n\n/* The magnitude"),
    # sign error
    "sign": ("for (int64_t jj = 0; jj < V; ++jj) cb[jj] += av * (double)bb[jj];\n            }\n        }\n    }\n    return 0;\n}\n\n/* The magnitude",
             "for (int64_t jj = 0; jj < V; ++jj) cb[jj] -= av * (double)bb[jj];\n            }\n        }\n    }\n    return 0;\n}\n\n/* The magnitude"),
    # compressed rows read in reverse (a transposed / mis-strided operand)
    "reversed_rows": ("const float *brow = Bc + u * n;\n            const uint8_t *drow = idx + u * q;\n            for (int64_t b = 0; b < q; ++b) {\n                const double av = (double)",
                      "const float *brow = Bc + (w - 1 - u) * n;\n            const uint8_t *drow = idx + u * q;\n            for (int64_t b = 0; b < q; ++b) {\n                const double av = (double)"),
    # compressor keeps the smallest rows
    "keeps_smallest": ("if (best < 0 || score[o] > score[best]) best = o;",
                       "if (best < 0 || score[o] < score[best]) best = o;"),
    # compressor breaks ties toward the larger offset
    "ties_to_larger": ("if (best < 0 || score[o] > score[best]) best = o;",
                       "if (best < 0 || score[o] >= score[best]) best = o;"),
    # epilogue: Eq. 1's factor dropped, GELU's argument unscaled, leaky ReLU
    "alpha_dropped": ("double y = alpha * C[i * n + j];", "double y = C[i * n + j];"),
    "gelu_scale": ("erf(y / sqrt(2.0))", "erf(y / 2.0)"),
    "leaky_relu": ("y = y > 0.0 ? y : 0.0;", "y = y > 0.0 ? y : 0.01 * y;"),
    # Eq. 2: the dense product drops its last k-row or reads B's rows reversed;
    # W loses the absolute value or divides by m + n
    "dense_dropped_term": ("for (int64_t kk = 0; kk < k; ++kk) {\n            const double av = (double)a[kk];",
                           "for (int64_t kk = 0; kk + 1 < k; ++kk) {\n            const double av = (double)a[kk];"),
    "dense_reversed_rows": ("const float *brow = B + kk * n;", "const float *brow = B + (k - 1 - kk) * n;"),
    "confusion_signed": ("W[i * n + j] = fabs(Cs[i * n + j] - C[i * n + j]) / mn;",
                         "W[i * n + j] = (Cs[i * n + j] - C[i * n + j]) / mn;"),
    "confusion_norm": ("const double mn = (double)m * (double)n;", "const double mn = (double)m + (double)n;"),
}
EPILOGUE_MUTANTS = ("alpha_dropped", "gelu_scale", "leaky_relu")
EQ2_MUTANTS = ("dense_dropped_term", "dense_reversed_rows", "confusion_signed", "confusion_norm")


class _Lib:
    def __init__(self, path):
        L = ctypes.CDLL(path)
        F = ctypes.POINTER(ctypes.c_float)
        D = ctypes.POINTER(ctypes.c_double)
        U8 = ctypes.POINTER(ctypes.c_uint8)
        I64, I = ctypes.c_int64, ctypes.c_int
        L.oracle_spmm.argtypes = [F, F, U8, D, I64, I64, I64, I, I, I]
        L.oracle_compress.argtypes = [F, I64, I64, I, I, I, F, U8]
        L.oracle_epilogue.argtypes = [D, I64, I64, ctypes.c_double, F, I]
        L.oracle_dense.argtypes = [F, F, D, I64, I64, I64]
        L.oracle_confusion.argtypes = [D, D, D, I64, I64]
        self.L, self.F, self.D, self.U8 = L, F, D, U8

    def dense(self, A, B):
        A = np.ascontiguousarray(A, np.float32)
        B = np.ascontiguousarray(B, np.float32)
        C = np.zeros((A.shape[0], B.shape[1]), np.float64)
        self.L.oracle_dense(A.ctypes.data_as(self.F), B.ctypes.data_as(self.F), C.ctypes.data_as(self.D),
                            A.shape[0], B.shape[1], A.shape[1])
        return C

    def confusion(self, Cs, C):
        Cs = np.ascontiguousarray(Cs, np.float64)
        C = np.ascontiguousarray(C, np.float64)
        W = np.zeros(C.shape, np.float64)
        self.L.oracle_confusion(Cs.ctypes.data_as(self.D), C.ctypes.data_as(self.D), W.ctypes.data_as(self.D),
                                C.shape[0], C.shape[1])
        return W

    def epilogue(self, C, alpha, act):
        out = np.ascontiguousarray(C, np.float64).copy()
        self.L.oracle_epilogue(out.ctypes.data_as(self.D), out.shape[0], out.shape[1], alpha, None, act)
        return out

    def compress(self, B, N, M, V):
        k, n = B.shape
        B = np.ascontiguousarray(B, np.float32)
        Bc = np.zeros(((k // M) * N, n), np.float32)
        idx = np.zeros(((k // M) * N, n // V), np.uint8)
        self.L.oracle_compress(B.ctypes.data_as(self.F), k, n, N, M, V,
                               Bc.ctypes.data_as(self.F), idx.ctypes.data_as(self.U8))
        return Bc, idx

    def spmm(self, A, Bc, idx, m, n, k, N, M, V):
        # one spare row after A so that a mutant reading past a row stays in bounds
        Ap = np.zeros((m + 2, k), np.float32)
        Ap[:m] = A
        C = np.zeros((m, n), np.float64)
        self.L.oracle_spmm(Ap.ctypes.data_as(self.F), np.ascontiguousarray(Bc).ctypes.data_as(self.F),
                           np.ascontiguousarray(idx).ctypes.data_as(self.U8),
                           C.ctypes.data_as(self.D), m, n, k, N, M, V)
        return C


def _dense_sequential(A, B):
    C = np.zeros((A.shape[0], B.shape[1]))
    for kk in range(A.shape[1]):
        C += np.outer(A[:, kk].astype(np.float64), B[kk].astype(np.float64))
    return C


def failing_pins(lib):
    """Names of the pins that the given oracle build fails."""
    fails = []
    # brute force against the dense sequential product
    for (m, k, n, N, M, V) in [(7, 16, 16, 2, 4, 4), (9, 64, 64, 16, 32, 32), (5, 64, 32, 4, 32, 8)]:
        A, Bp, _ = make_inputs(m, k, n, N, M, V, seed=31 + k)
        Bc, idx = lib.compress(Bp, N, M, V)
        if not np.array_equal(lib.spmm(A, Bc, idx, m, n, k, N, M, V), _dense_sequential(A, Bp)):
            fails.append("brute_force")
            break
    # power-of-two bit mask encoding
    k, n, N, M, V = 48, 16, 2, 4, 4
    _, _, mask = make_inputs(1, k, n, N, M, V, seed=21)
    A = (2.0 ** np.arange(k))[None, :].astype(np.float32)
    Bc, idx = lib.compress(mask.astype(np.float32), N, M, V)
    C = lib.spmm(A, Bc, idx, 1, n, k, N, M, V)
    if any(C[0, j] != float(sum(1 << kk for kk in range(k) if mask[kk, j])) for j in range(n)):
        fails.append("bitmask")
    # hand example (golden)
    g = json.load(open(os.path.join(GOLDEN, "fig1_hand_example.json")))
    Bc = np.full((4, 8), 1.0, np.float32)
    C = lib.spmm(np.array(g["A"], np.float32), Bc, np.array(g["idx"], np.uint8), 2, 8, 8, 2, 4, 4)
    if not np.array_equal(C, np.array(g["C_expected"], np.float64)):
        fails.append("hand_example")
    # compress recovers the generator's mask (continuous values)
    k, n, N, M, V = 64, 64, 4, 32, 8
    _, Bp, mask = make_inputs(1, k, n, N, M, V, seed=8)
    Bc, idx = lib.compress(Bp, N, M, V)
    rec = np.zeros((k, n // V), bool)
    for u in range(idx.shape[0]):
        for b in range(idx.shape[1]):
            rec[(u // N) * M + idx[u, b], b] = True
    if not np.array_equal(np.repeat(rec, V, axis=1), mask):
        fails.append("mask_recovery")
    # ties resolve to the smaller offset
    _, idx = lib.compress(np.ones((8, 4), np.float32), 2, 4, 2)
    if not np.array_equal(idx, np.array([[0, 0], [1, 1], [0, 0], [1, 1]], np.uint8)):
        fails.append("ties")
    # epilogue: alpha scales exactly, ReLU clamps at zero, GELU matches
    # scipy's normal CDF
    from scipy.stats import norm
    C = np.linspace(-4, 4, 33)[None, :]
    if not np.array_equal(lib.epilogue(C, 4.0, 0), 4.0 * C):
        fails.append("epilogue_alpha")
    if not np.array_equal(lib.epilogue(C, 1.0, 1), np.maximum(C, 0.0)):
        fails.append("epilogue_relu")
    if not np.allclose(lib.epilogue(C, 1.0, 2), C * norm.cdf(C), rtol=1e-13, atol=1e-15):
        fails.append("epilogue_gelu")
    # Eq. 2: the dense product against the sequential product, and the
    # hand-worked confusion matrix (golden)
    rng = np.random.default_rng(12)
    A = rng.uniform(-1, 1, (5, 12)).astype(np.float32)
    B = rng.uniform(-1, 1, (12, 7)).astype(np.float32)
    if not np.array_equal(lib.dense(A, B), _dense_sequential(A, B)):
        fails.append("dense_brute_force")
    g = json.load(open(os.path.join(GOLDEN, "eq2_hand_example.json")))
    A, B = np.array(g["A"], np.float32), np.array(g["B"], np.float32)
    N, M, V, m, k, n = g["N"], g["M"], g["V"], g["m"], g["k"], g["n"]
    Bc, idx = lib.compress(B, N, M, V)
    Cs = lib.epilogue(lib.spmm(A, Bc, idx, m, n, k, N, M, V), M / N, 0)
    if not np.array_equal(lib.confusion(Cs, lib.dense(A, B)), np.array(g["W_expected"], np.float64)):
        fails.append("eq2_hand_example")
    return fails


@pytest.fixture(scope="module")
def source():
    return open(SRC).read()


def test_unmutated_oracle_passes_all_pins(tmp_path, source):
    path = build(out=str(tmp_path / "liboracle_copy.so"))
    assert failing_pins(_Lib(path)) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_every_planted_mistake_is_caught(tmp_path, source, name):
    old, new = MUTANTS[name]
    # the first occurrence of each site lies in oracle_spmm (or, for the
    # selection sites, in oracle_compress); only that one is changed
    at = source.find(old)
    assert at >= 0, f"mutation site for {name} not found"
    if name not in ("keeps_smallest", "ties_to_larger") + EPILOGUE_MUTANTS + EQ2_MUTANTS:
        assert at < source.index("int oracle_bound(")
    src = tmp_path / f"mutant_{name}.c"
    src.write_text(source.replace(old, new, 1))
    path = build(out=str(tmp_path / f"libmutant_{name}.so"), src=str(src))
    assert failing_pins(_Lib(path)), f"no pin caught mutant {name}"
