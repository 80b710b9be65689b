"""CPU oracle for vector-wise N:M SpMM (NM-SpMM, arXiv 2503.01253, Sec. II-A, Eq. 1).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg may import this package; the product path never does.  It is
a thin ctypes wrapper around ``nm_oracle.c`` (plain C, fp64) plus the parity
checker.  It imports nothing from the HIP package and shares no code with it.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .build import LIB_PATH, build

__all__ = [
    "build", "lib", "spmm", "bound", "compress", "decompress", "validate", "epilogue",
    "dense", "confusion", "set_threads", "max_threads", "check", "CheckResult", "PARITY_RTOL",
]

# Parity bar: |C_gpu - C_ref| <= PARITY_RTOL * sum_k |A_ik| |B_kj| for every
# element, and every element finite.
PARITY_RTOL = 1e-5

_lib = None
_F = ctypes.POINTER(ctypes.c_float)
_D = ctypes.POINTER(ctypes.c_double)
_U8 = ctypes.POINTER(ctypes.c_uint8)
_I64 = ctypes.c_int64
_I = ctypes.c_int


def lib():
    """Load liboracle_nm.so, building it first if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        L.oracle_spmm.argtypes = [_F, _F, _U8, _D, _I64, _I64, _I64, _I, _I, _I]
        L.oracle_bound.argtypes = [_F, _F, _U8, _D, _I64, _I64, _I64, _I, _I, _I]
        L.oracle_compress.argtypes = [_F, _I64, _I64, _I, _I, _I, _F, _U8]
        L.oracle_decompress.argtypes = [_F, _U8, _I64, _I64, _I, _I, _I, _F]
        L.oracle_validate.argtypes = [_U8, _I64, _I64, _I, _I, _I]
        L.oracle_shape_ok.argtypes = [_I64, _I64, _I64, _I, _I, _I]
        L.oracle_set_threads.argtypes = [_I]
        L.oracle_epilogue.argtypes = [_D, _I64, _I64, ctypes.c_double, _F, _I]
        L.oracle_epilogue.restype = _I
        L.oracle_dense.argtypes = [_F, _F, _D, _I64, _I64, _I64]
        L.oracle_dense.restype = _I
        L.oracle_confusion.argtypes = [_D, _D, _D, _I64, _I64]
        L.oracle_confusion.restype = _I
        for f in (L.oracle_spmm, L.oracle_bound, L.oracle_compress, L.oracle_decompress,
                  L.oracle_validate, L.oracle_shape_ok, L.oracle_max_threads):
            f.restype = _I
        L.oracle_set_threads.restype = None
        _lib = L
    return _lib


def _p(a, ty):
    return a.ctypes.data_as(ty)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _u8(a):
    return np.ascontiguousarray(a, dtype=np.uint8)


def spmm(A, Bc, idx, m, n, k, N, M, V):
    """Eq. 1 (read without the M/N factor, window base floor(u/N)*M): fp64 C."""
    A, Bc, idx = _f32(A), _f32(Bc), _u8(idx)
    C = np.empty((m, n), dtype=np.float64)
    rc = lib().oracle_spmm(_p(A, _F), _p(Bc, _F), _p(idx, _U8), _p(C, _D), m, n, k, N, M, V)
    if rc:
        raise ValueError(f"oracle_spmm: bad shape m={m} n={n} k={k} N={N} M={M} V={V}")
    return C


def bound(A, Bc, idx, m, n, k, N, M, V):
    """sum_u |A[i][col(u, j)]| |Bc[u][j]| in fp64 (the tolerance scale)."""
    A, Bc, idx = _f32(A), _f32(Bc), _u8(idx)
    C = np.empty((m, n), dtype=np.float64)
    rc = lib().oracle_bound(_p(A, _F), _p(Bc, _F), _p(idx, _U8), _p(C, _D), m, n, k, N, M, V)
    if rc:
        raise ValueError("oracle_bound: bad shape")
    return C


def compress(B, N, M, V):
    """Dense pruned (or unpruned) B -> (Bc, idx), Sec. II-A."""
    B = _f32(B)
    k, n = B.shape
    w = (k // M) * N if M else 0
    q = n // V if V else 0
    Bc = np.empty((w, n), dtype=np.float32)
    idx = np.empty((w, q), dtype=np.uint8)
    rc = lib().oracle_compress(_p(B, _F), k, n, N, M, V, _p(Bc, _F), _p(idx, _U8))
    if rc:
        raise ValueError(f"oracle_compress: bad shape k={k} n={n} N={N} M={M} V={V}")
    return Bc, idx


def decompress(Bc, idx, k, n, N, M, V):
    Bc, idx = _f32(Bc), _u8(idx)
    B = np.empty((k, n), dtype=np.float32)
    rc = lib().oracle_decompress(_p(Bc, _F), _p(idx, _U8), k, n, N, M, V, _p(B, _F))
    if rc:
        raise ValueError("oracle_decompress: bad shape")
    return B


def validate(idx, k, n, N, M, V):
    """0 valid, 1 bad shape, 2 offset >= M, 3 not strictly increasing."""
    idx = _u8(idx)
    return int(lib().oracle_validate(_p(idx, _U8), k, n, N, M, V))


ACTS = {"none": 0, "relu": 1, "gelu": 2}


def epilogue(C, alpha=1.0, bias=None, act="none"):
    """act(alpha * C + bias[j]) on an fp64 product (Eq. 1's M/N factor is
    alpha = M/N); returns a new fp64 array."""
    out = np.ascontiguousarray(C, dtype=np.float64).copy()
    m, n = out.shape
    b = None if bias is None else _f32(bias)
    if b is not None and b.shape != (n,):
        raise ValueError("bias must have n entries")
    st = lib().oracle_epilogue(_p(out, _D), m, n, float(alpha),
                               None if b is None else _p(b, _F), ACTS[act])
    if st != 0:
        raise ValueError(f"oracle_epilogue failed ({st})")
    return out


def dense(A, B):
    """C = A * B with the unpruned B (the dense output of Eq. 2), fp64."""
    A, B = _f32(A), _f32(B)
    m, k = A.shape
    k2, n = B.shape
    if k2 != k:
        raise ValueError(f"inner sizes differ: {k} and {k2}")
    C = np.empty((m, n), dtype=np.float64)
    if lib().oracle_dense(_p(A, _F), _p(B, _F), _p(C, _D), m, n, k):
        raise ValueError("oracle_dense: bad shape")
    return C


def confusion(Cs, C):
    """Eq. 2: W = |Cs - C| / (m*n) in fp64, Cs the N:M output with Eq. 1's
    M/N factor and C the dense output."""
    Cs = np.ascontiguousarray(Cs, dtype=np.float64)
    C = np.ascontiguousarray(C, dtype=np.float64)
    if Cs.shape != C.shape or Cs.ndim != 2:
        raise ValueError(f"shape mismatch {Cs.shape} {C.shape}")
    m, n = C.shape
    W = np.empty((m, n), dtype=np.float64)
    if lib().oracle_confusion(_p(Cs, _D), _p(C, _D), _p(W, _D), m, n):
        raise ValueError("oracle_confusion: bad shape")
    return W


def set_threads(t: int) -> None:
    lib().oracle_set_threads(int(t))


def max_threads() -> int:
    return int(lib().oracle_max_threads())


class CheckResult:
    def __init__(self, ok, worst_ratio, worst_index, n_bad, n_nonfinite):
        self.ok = ok
        self.worst_ratio = worst_ratio
        self.worst_index = worst_index
        self.n_bad = n_bad
        self.n_nonfinite = n_nonfinite

    def __bool__(self):
        return self.ok

    def __repr__(self):
        return (f"CheckResult(ok={self.ok}, worst_ratio={self.worst_ratio:.3e}, "
                f"worst_index={self.worst_index}, n_bad={self.n_bad}, "
                f"n_nonfinite={self.n_nonfinite})")


def check(C_test, C_ref, Bnd, rtol=PARITY_RTOL):
    """Element-wise parity: finite, and |C_test - C_ref| <= rtol * Bnd.

    ``worst_ratio`` is max |err| / Bnd over elements with Bnd > 0 (elements
    with Bnd == 0 must match exactly)."""
    C_test = np.asarray(C_test, dtype=np.float64)
    C_ref = np.asarray(C_ref, dtype=np.float64)
    Bnd = np.asarray(Bnd, dtype=np.float64)
    if C_test.shape != C_ref.shape or C_ref.shape != Bnd.shape:
        raise ValueError(f"shape mismatch {C_test.shape} {C_ref.shape} {Bnd.shape}")
    finite = np.isfinite(C_test)
    n_nonfinite = int(C_test.size - np.count_nonzero(finite))
    err = np.abs(np.where(finite, C_test, np.inf) - C_ref)
    bad = ~(err <= rtol * Bnd)
    n_bad = int(np.count_nonzero(bad))
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(Bnd > 0, err / np.where(Bnd > 0, Bnd, 1.0),
                         np.where(err == 0, 0.0, np.inf))
    if ratio.size:
        flat = int(np.argmax(ratio))
        worst = float(ratio.reshape(-1)[flat])
        worst_index = np.unravel_index(flat, ratio.shape)
    else:
        worst, worst_index = 0.0, None
    return CheckResult(n_bad == 0 and n_nonfinite == 0, worst, worst_index, n_bad, n_nonfinite)
