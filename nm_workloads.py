"""Seeded synthetic inputs for vector-wise N:M SpMM, shared by the tests, the
benchmark and the smoke check.

This module draws random numbers and builds the dense pruned weight; it holds
none of the method's arithmetic (no compression, no product).  Both the oracle
and the HIP path receive exactly the arrays made here.

Recipe (mirrors the workloads of Sec. IV: fp32 operands, the paper's sparsity
levels 50 / 62.5 / 75 / 87.5 % at M = 32, and LLM-shaped layers):
  1. A (m x k) from the named distribution, fp32.
  2. B (k x n) from the named distribution, fp32.
  3. For every (group g < k/M, column block b < n/V) a uniformly random
     N-subset of the M offsets, drawn as the first N entries of an argsort of
     M uniform numbers.
  4. B_pruned = B where kept, else 0.
Distributions: "uniform" = U[-1, 1] for A and B; "normal" = A ~ N(0, 1),
B ~ N(0, 0.02^2) (standard deviation 0.02).  Generation uses numpy's PCG64
``default_rng(seed)``, platform-stable.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Run:
    name: str
    m: int
    k: int
    n: int
    N: int
    M: int
    V: int
    dist: str
    seed: int

    @property
    def w(self) -> int:
        return (self.k // self.M) * self.N

    @property
    def q(self) -> int:
        return self.n // self.V

    @property
    def useful_flops(self) -> float:
        """2 m n k N / M: the multiply-adds the sparse product must do."""
        return 2.0 * self.m * self.n * self.w

    @property
    def alg_bytes(self) -> float:
        """A read once, Bc read once, idx (1 byte per entry) read once, C written once."""
        return 4.0 * self.m * self.k + 4.0 * self.w * self.n + self.w * self.q + 4.0 * self.m * self.n

    def describe(self) -> str:
        return (f"{self.name}: m={self.m} k={self.k} n={self.n} {self.N}:{self.M} V={self.V} "
                f"{self.dist} seed={self.seed}")


# The five workload families: a small square case, the paper's 4096^3 case at
# 50 / 75 / 87.5 % sparsity (Sec. IV-B, IV-E), an LLM MLP up-projection shape
# (k = 4096, n = 11008, m = 2048 tokens; the paper's Llama-layer set of Sec.
# IV-A is not published, this shape stands in for it) and decode-like skinny
# products (m = 16 / 64 / 128 at k = n = 8192).
RUNS = {
    "R1": Run("R1", 256, 256, 256, 16, 32, 32, "uniform", 1001),
    "R2": Run("R2", 4096, 4096, 4096, 16, 32, 32, "uniform", 1002),
    "R3a": Run("R3a", 4096, 4096, 4096, 8, 32, 32, "uniform", 1003),
    "R3b": Run("R3b", 4096, 4096, 4096, 8, 32, 64, "uniform", 1004),
    "R3c": Run("R3c", 4096, 4096, 4096, 4, 32, 32, "uniform", 1005),
    "R3d": Run("R3d", 4096, 4096, 4096, 4, 32, 64, "uniform", 1006),
    "R4": Run("R4", 2048, 4096, 11008, 8, 32, 32, "normal", 1007),
    "R5a": Run("R5a", 16, 8192, 8192, 4, 32, 64, "normal", 1008),
    "R5b": Run("R5b", 64, 8192, 8192, 4, 32, 64, "normal", 1009),
    "R5c": Run("R5c", 128, 8192, 8192, 4, 32, 64, "normal", 1010),
}


# The kernel-family sweep of Sec. IV-C: the six small / medium / large shapes
# of the paper's matrix-size table (A-F) at the five sparsity levels of
# Sec. IV-B and IV-C, 0 % (N = M = 32, the dense-equivalence point), 50 %,
# 62.5 %, 75 % and 87.5 %; V = 32, U[-1, 1].
TABLE_SHAPES = {
    "A": (512, 512, 512), "B": (512, 1024, 1024), "C": (512, 2048, 2048),
    "D": (1024, 2048, 2048), "E": (2048, 4096, 4096), "F": (4096, 4096, 4096),
}
TABLE_LEVELS = (32, 16, 12, 8, 4)    # N at M = 32


def table_runs():
    """Runs of the shape x sparsity sweep, keyed "A-32" .. "F-4" (shape-N)."""
    out = {}
    for i, (label, (m, n, k)) in enumerate(TABLE_SHAPES.items()):
        for j, N in enumerate(TABLE_LEVELS):
            name = f"{label}-{N}"
            out[name] = Run(name, m, k, n, N, 32, 32, "uniform", 2000 + 10 * i + j)
    return out


def random_mask(rng: np.random.Generator, k: int, n: int, N: int, M: int, V: int) -> np.ndarray:
    """Boolean k x n mask: N kept rows per (window of M rows, block of V columns)."""
    G, q = k // M, n // V
    if G == 0 or q == 0:
        return np.zeros((k, n), dtype=bool)
    order = np.argsort(rng.random((G, q, M)), axis=-1)[..., :N]  # (G, q, N)
    keep = np.zeros((G, q, M), dtype=bool)
    np.put_along_axis(keep, order, True, axis=-1)
    # (G, q, M) -> (G, M, q) -> (k, q) -> repeat each block V times -> (k, n)
    rows = keep.transpose(0, 2, 1).reshape(k, q)
    return np.repeat(rows, V, axis=1)


def _draw(rng, dist, shape, role):
    if dist == "uniform":
        return rng.uniform(-1.0, 1.0, size=shape).astype(np.float32)
    if dist == "normal":
        x = rng.standard_normal(size=shape)
        return (x * (0.02 if role == "B" else 1.0)).astype(np.float32)
    if dist == "int":
        # small integers: every partial sum of the product is an exact fp32
        # integer as long as k * 8 * 8 < 2^24
        return rng.integers(-8, 9, size=shape).astype(np.float32)
    raise ValueError(f"unknown distribution {dist!r}")


def make_inputs(m: int, k: int, n: int, N: int, M: int, V: int, seed: int,
                dist: str = "uniform"):
    """Return (A, B_pruned, mask) as C-contiguous arrays (fp32, fp32, bool)."""
    rng = np.random.default_rng(seed)
    A = _draw(rng, dist, (m, k), "A")
    B = _draw(rng, dist, (k, n), "B")
    mask = random_mask(rng, k, n, N, M, V)
    if dist == "int":
        # kept entries must be non-zero so that the kept set is recoverable
        B = np.where(B == 0, np.float32(1), B)
    B_pruned = np.where(mask, B, np.float32(0)).astype(np.float32)
    return np.ascontiguousarray(A), np.ascontiguousarray(B_pruned), mask


def make_run(run: Run, m: int | None = None):
    """Inputs of a named run; ``m`` overrides the row count (A's first rows)."""
    A, Bp, mask = make_inputs(run.m, run.k, run.n, run.N, run.M, run.V, run.seed, run.dist)
    if m is not None:
        A = np.ascontiguousarray(A[:m])
    return A, Bp, mask
