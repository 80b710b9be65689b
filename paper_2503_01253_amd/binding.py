"""ctypes binding of libnmspmm.so: the C-ABI entry points under the same names.

Argument marshalling only.  Device buffers are PyTorch tensors (torch provides
HIP memory and streams); every step of the product runs in the library's HIP
kernels.  There is no fallback: if the library is not built, every call
raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .build import LIB_PATH

NMSPMM_OK = 0
NMSPMM_ERR_INVALID_ARG = 1
NMSPMM_ERR_UNSUPPORTED = 2
NMSPMM_ERR_HIP = 3
NMSPMM_ERR_SCRATCH = 4
NMSPMM_NOALLOC_SCRATCH_BYTES = 16 << 20

NMSPMM_ACT_NONE = 0
NMSPMM_ACT_RELU = 1
NMSPMM_ACT_GELU = 2
ACTS = {"none": NMSPMM_ACT_NONE, "relu": NMSPMM_ACT_RELU, "gelu": NMSPMM_ACT_GELU}

EXPORTS = (
    "nmspmm_bc_elems", "nmspmm_idx_bytes", "nmspmm_compress", "nmspmm_compress_device",
    "nmspmm_run", "nmspmm_run_ex", "nmspmm_run_ws", "nmspmm_workspace_bytes", "nmspmm_validate_idx",
    "nmspmm_status_string", "nmspmm_kernel_name", "nmspmm_kernel_name_ws",
    "nmspmm_run_tuned", "nmspmm_kernel_name_tuned", "nmspmm_workspace_bytes_tuned", "nmspmm_run_noalloc",
    "nmspmm_confusion",
)


class NmSpmmError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn}: {msg} (status {status})")
        self.status = status


_lib = None


def lib():
    """Load the built library.  torch is imported first so that the library
    binds to the HIP runtime torch already loaded (same soname), keeping
    torch's streams and allocations valid inside the library."""
    global _lib
    if _lib is None:
        _lib = load(LIB_PATH)
    return _lib


def load(path: str):
    """A ctypes handle on a build of the library at `path` (the product
    library, or its NaN-poisoned debug twin for the LDS race tests), with
    every entry point's signature declared."""
    import torch  # noqa: F401  (loads torch's libamdhip64 before ours)
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built: run `python -m paper_2503_01253_amd.build`")
    L = ctypes.CDLL(path)
    I64, I, P = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
    L.nmspmm_bc_elems.argtypes = [I64, I64, I, I]
    L.nmspmm_bc_elems.restype = I64
    L.nmspmm_idx_bytes.argtypes = [I64, I64, I, I, I]
    L.nmspmm_idx_bytes.restype = I64
    L.nmspmm_compress.argtypes = [P, I64, I64, I, I, I, P, P]
    L.nmspmm_compress.restype = I
    L.nmspmm_run.argtypes = [P, P, P, P, I64, I64, I64, I, I, I, P]
    L.nmspmm_run.restype = I
    L.nmspmm_validate_idx.argtypes = [P, I64, I64, I, I, I]
    L.nmspmm_validate_idx.restype = I
    L.nmspmm_status_string.argtypes = [I]
    L.nmspmm_status_string.restype = ctypes.c_char_p
    L.nmspmm_kernel_name.argtypes = [I64, I64, I64, I, I, I]
    L.nmspmm_kernel_name.restype = ctypes.c_char_p
    L.nmspmm_kernel_name_ws.argtypes = [I64, I64, I64, I, I, I]
    L.nmspmm_kernel_name_ws.restype = ctypes.c_char_p
    L.nmspmm_run_ex.argtypes = [P, P, P, P, I64, I64, I64, I, I, I, ctypes.c_float, P, I, P]
    L.nmspmm_run_ex.restype = I
    L.nmspmm_compress_device.argtypes = [P, I64, I64, I, I, I, P, P, P]
    L.nmspmm_compress_device.restype = I
    L.nmspmm_run_ws.argtypes = [P, P, P, P, I64, I64, I64, I, I, I, ctypes.c_float, P, I, P,
                                ctypes.c_size_t, P]
    L.nmspmm_run_ws.restype = I
    L.nmspmm_workspace_bytes.argtypes = [I64, I64, I64, I, I, I]
    L.nmspmm_workspace_bytes.restype = I64
    L.nmspmm_run_tuned.argtypes = [P, P, P, P, I64, I64, I64, I, I, I, ctypes.c_float, P, I, P,
                                   ctypes.c_size_t, ctypes.c_char_p, P]
    L.nmspmm_run_tuned.restype = I
    L.nmspmm_kernel_name_tuned.argtypes = [I64, I64, I64, I, I, I, I, ctypes.c_char_p]
    L.nmspmm_kernel_name_tuned.restype = ctypes.c_char_p
    L.nmspmm_workspace_bytes_tuned.argtypes = [I64, I64, I64, I, I, I, ctypes.c_char_p]
    L.nmspmm_workspace_bytes_tuned.restype = I64
    L.nmspmm_run_noalloc.argtypes = [P, P, P, P, I64, I64, I64, I, I, I, ctypes.c_float, P, I, P]
    L.nmspmm_run_noalloc.restype = I
    L.nmspmm_confusion.argtypes = [P, P, P, I64, I64, P]
    L.nmspmm_confusion.restype = I
    return L


def nmspmm_status_string(status: int) -> str:
    return lib().nmspmm_status_string(int(status)).decode()


def _check(fn, status):
    if status != NMSPMM_OK:
        raise NmSpmmError(fn, status, nmspmm_status_string(status))


def nmspmm_bc_elems(k: int, n: int, N: int, M: int) -> int:
    return int(lib().nmspmm_bc_elems(k, n, N, M))


def nmspmm_idx_bytes(k: int, n: int, N: int, M: int, V: int) -> int:
    return int(lib().nmspmm_idx_bytes(k, n, N, M, V))


def tuning_string(tuning) -> bytes | None:
    """The tuning overrides of the *_tuned entry points as the library's
    "KEY=VALUE,..." string (a dict or a string; None or empty: no override).
    For tile sweeps and forced-variant tests only."""
    if not tuning:
        return None
    if isinstance(tuning, dict):
        tuning = ",".join(f"{k}={v}" for k, v in tuning.items())
    return tuning.encode()


def nmspmm_kernel_name(m: int, n: int, k: int, N: int, M: int, V: int, tuning=None) -> str:
    if tuning:
        return lib().nmspmm_kernel_name_tuned(m, n, k, N, M, V, 0, tuning_string(tuning)).decode()
    return lib().nmspmm_kernel_name(m, n, k, N, M, V).decode()


def nmspmm_kernel_name_ws(m: int, n: int, k: int, N: int, M: int, V: int, tuning=None) -> str:
    if tuning:
        return lib().nmspmm_kernel_name_tuned(m, n, k, N, M, V, 1, tuning_string(tuning)).decode()
    return lib().nmspmm_kernel_name_ws(m, n, k, N, M, V).decode()


def nmspmm_compress(B_dense: np.ndarray, N: int, M: int, V: int):
    """Host packer: dense (pruned) B, k x n fp32 -> (Bc, idx) numpy arrays."""
    B = np.ascontiguousarray(B_dense, dtype=np.float32)
    if B.ndim != 2:
        raise ValueError("B_dense must be 2-D")
    k, n = B.shape
    nbc = nmspmm_bc_elems(k, n, N, M)
    nidx = nmspmm_idx_bytes(k, n, N, M, V)
    if nbc < 0 or nidx < 0:
        raise NmSpmmError("nmspmm_compress", NMSPMM_ERR_INVALID_ARG,
                          f"invalid shape k={k} n={n} N={N} M={M} V={V}")
    w = (k // M) * N
    Bc = np.empty((w, n), dtype=np.float32)
    idx = np.empty((w, n // V), dtype=np.uint8)
    st = lib().nmspmm_compress(B.ctypes.data, k, n, N, M, V, Bc.ctypes.data, idx.ctypes.data)
    _check("nmspmm_compress", st)
    return Bc, idx


def nmspmm_validate_idx(idx: np.ndarray, k: int, n: int, N: int, M: int, V: int) -> int:
    """Returns the status code (0 = valid pattern)."""
    d = np.ascontiguousarray(idx, dtype=np.uint8)
    return int(lib().nmspmm_validate_idx(d.ctypes.data, k, n, N, M, V))


def nmspmm_run_ptr(A: int, Bc: int, idx: int, C: int, m: int, n: int, k: int,
                   N: int, M: int, V: int, stream: int) -> int:
    """Raw entry point: device addresses and a hipStream_t as integers.
    Returns the status code."""
    return int(lib().nmspmm_run(A, Bc, idx, C, m, n, k, N, M, V, stream))


def _check_tensors(torch, C, specs):
    for name, t, dt, numel in specs:
        if not isinstance(t, torch.Tensor) or t.dtype != dt or not t.is_cuda or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous CUDA tensor of {dt}")
        if t.device != C.device:
            raise ValueError(f"{name} is on {t.device}, {C.device} expected")
        if t.numel() != numel:
            raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")


def nmspmm_run(A, Bc, idx, C, m: int, n: int, k: int, N: int, M: int, V: int, stream=None, tuning=None):
    """C = A * B_pruned on the GPU, asynchronously on ``stream`` (a
    torch.cuda.Stream; default: torch's current stream).  A (m x k), Bc
    (w x n), C (m x n) are contiguous fp32 CUDA tensors, idx (w x q) a
    contiguous uint8 CUDA tensor, all on one device.  ``tuning`` (sweeps and
    tests only) routes the call through nmspmm_run_tuned."""
    return nmspmm_run_ex(A, Bc, idx, C, m, n, k, N, M, V, stream=stream, tuning=tuning, _name="nmspmm_run")


def nmspmm_workspace_bytes(m: int, n: int, k: int, N: int, M: int, V: int, tuning=None) -> int:
    """Workspace bytes nmspmm_run_ws can use for this shape (0: none; -1: bad shape)."""
    if tuning:
        return int(lib().nmspmm_workspace_bytes_tuned(m, n, k, N, M, V, tuning_string(tuning)))
    return int(lib().nmspmm_workspace_bytes(m, n, k, N, M, V))


def nmspmm_run_ws(A, Bc, idx, C, m: int, n: int, k: int, N: int, M: int, V: int, workspace,
                  alpha: float = 1.0, bias=None, act: str = "none", stream=None, tuning=None):
    """nmspmm_run_ex with a split-k workspace: a uint8 CUDA tensor of at least
    nmspmm_workspace_bytes bytes, 256-byte aligned (or None, or smaller: the
    call runs as nmspmm_run_ex)."""
    return nmspmm_run_ex(A, Bc, idx, C, m, n, k, N, M, V, alpha, bias, act, stream, tuning=tuning,
                         _name="nmspmm_run_ws", _workspace=workspace)


def nmspmm_run_noalloc(A, Bc, idx, C, m: int, n: int, k: int, N: int, M: int, V: int,
                       alpha: float = 1.0, bias=None, act: str = "none", stream=None):
    """nmspmm_run_ws with the library's static per-device scratch array as the
    workspace (for callers that cannot allocate); raises NmSpmmError with
    NMSPMM_ERR_SCRATCH when the shape needs more than
    NMSPMM_NOALLOC_SCRATCH_BYTES.  Calls that overlap on one device race."""
    return nmspmm_run_ex(A, Bc, idx, C, m, n, k, N, M, V, alpha, bias, act, stream,
                         _name="nmspmm_run_noalloc")


def nmspmm_run_ex(A, Bc, idx, C, m: int, n: int, k: int, N: int, M: int, V: int,
                  alpha: float = 1.0, bias=None, act: str = "none", stream=None, tuning=None,
                  _name: str = "nmspmm_run_ex", _workspace=None):
    """C = act(alpha * (A * B_pruned) + bias) on the GPU (alpha = M/N is Eq. 1's
    factor; bias an n-element fp32 CUDA tensor or None; act "none", "relu" or
    "gelu").  Tensors and stream as for nmspmm_run; ``tuning`` as there."""
    import torch
    L = lib()
    w = (k // M) * N if M > 0 else 0
    q = n // V if V > 0 else 0
    specs = [("A", A, torch.float32, m * k), ("Bc", Bc, torch.float32, w * n),
             ("idx", idx, torch.uint8, w * q), ("C", C, torch.float32, m * n)]
    if bias is not None:
        specs.append(("bias", bias, torch.float32, n))
    if _workspace is not None:   # any size: too small means no workspace
        specs.append(("workspace", _workspace, torch.uint8, _workspace.numel()))
    _check_tensors(torch, C, specs)
    if act not in ACTS:
        raise ValueError(f"act must be one of {sorted(ACTS)}")
    if stream is None:
        stream = torch.cuda.current_stream(C.device)
    with torch.cuda.device(C.device):
        if tuning:
            st = L.nmspmm_run_tuned(A.data_ptr(), Bc.data_ptr(), idx.data_ptr(), C.data_ptr(),
                                    m, n, k, N, M, V, float(alpha),
                                    None if bias is None else bias.data_ptr(), ACTS[act],
                                    None if _workspace is None else _workspace.data_ptr(),
                                    0 if _workspace is None else _workspace.numel(),
                                    tuning_string(tuning), stream.cuda_stream)
            _name = "nmspmm_run_tuned"
        elif _name == "nmspmm_run_noalloc":
            st = L.nmspmm_run_noalloc(A.data_ptr(), Bc.data_ptr(), idx.data_ptr(), C.data_ptr(),
                                      m, n, k, N, M, V, float(alpha),
                                      None if bias is None else bias.data_ptr(), ACTS[act], stream.cuda_stream)
        elif _name == "nmspmm_run":
            st = L.nmspmm_run(A.data_ptr(), Bc.data_ptr(), idx.data_ptr(), C.data_ptr(),
                              m, n, k, N, M, V, stream.cuda_stream)
        elif _name == "nmspmm_run_ws":
            st = L.nmspmm_run_ws(A.data_ptr(), Bc.data_ptr(), idx.data_ptr(), C.data_ptr(),
                                 m, n, k, N, M, V, float(alpha),
                                 None if bias is None else bias.data_ptr(), ACTS[act],
                                 None if _workspace is None else _workspace.data_ptr(),
                                 0 if _workspace is None else _workspace.numel(), stream.cuda_stream)
        else:
            st = L.nmspmm_run_ex(A.data_ptr(), Bc.data_ptr(), idx.data_ptr(), C.data_ptr(),
                                 m, n, k, N, M, V, float(alpha),
                                 None if bias is None else bias.data_ptr(), ACTS[act],
                                 stream.cuda_stream)
    _check(_name, st)
    return C


def nmspmm_compress_device(B_dense, Bc, idx, N: int, M: int, V: int, stream=None):
    """Device packer: B_dense (k x n fp32 CUDA tensor) -> Bc (w x n fp32) and
    idx (w x q uint8), caller-allocated CUDA tensors, asynchronously on
    ``stream`` (default: torch's current stream)."""
    import torch
    if B_dense.dim() != 2:
        raise ValueError("B_dense must be 2-D")
    k, n = B_dense.shape
    w = (k // M) * N if M > 0 else 0
    q = n // V if V > 0 else 0
    _check_tensors(torch, B_dense, [("B_dense", B_dense, torch.float32, k * n),
                                    ("Bc", Bc, torch.float32, w * n), ("idx", idx, torch.uint8, w * q)])
    if stream is None:
        stream = torch.cuda.current_stream(B_dense.device)
    with torch.cuda.device(B_dense.device):
        st = lib().nmspmm_compress_device(B_dense.data_ptr(), k, n, N, M, V, Bc.data_ptr(),
                                          idx.data_ptr(), stream.cuda_stream)
    _check("nmspmm_compress_device", st)
    return Bc, idx


def nmspmm_confusion(C_sparse, C_dense, W, stream=None):
    """Eq. 2's confusion matrix W = |C_sparse - C_dense| / (m*n) on the GPU,
    asynchronously on ``stream`` (default: torch's current stream).
    C_sparse (Eq. 1's output with its M/N factor, e.g. from nmspmm_run_ex with
    alpha = M/N), C_dense (the product with the unpruned B) and W are
    contiguous m x n fp32 CUDA tensors on one device; W may be C_sparse or
    C_dense itself."""
    import torch
    if C_dense.dim() != 2:
        raise ValueError("C_dense must be 2-D")
    m, n = C_dense.shape
    _check_tensors(torch, W, [("C_sparse", C_sparse, torch.float32, m * n),
                              ("C_dense", C_dense, torch.float32, m * n), ("W", W, torch.float32, m * n)])
    if stream is None:
        stream = torch.cuda.current_stream(W.device)
    with torch.cuda.device(W.device):
        st = lib().nmspmm_confusion(C_sparse.data_ptr(), C_dense.data_ptr(), W.data_ptr(), m, n,
                                    stream.cuda_stream)
    _check("nmspmm_confusion", st)
    return W
