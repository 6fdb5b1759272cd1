"""Seeded synthetic CSR workloads shared by the oracle side and the GPU side.

Only input generation lives here (no SpGEMM arithmetic). Matrices are returned
as :class:`CSR` holding numpy arrays: ``row_ptr`` int64 (n_rows+1), ``col``
int32 (int64 for :func:`wide`; sorted, unique within a row) and ``val``
float64.

The five benchmark workloads are named in :data:`CONFIGS`; they stand in for
the paper's R-MAT pairs and SuiteSparse set (Section IV-A), which are not
available here.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB = os.path.join(_HERE, "libgmwork.so")

VALUE_MODES = {"u01": 0, "pm1": 1, "int3": 2, "ones": 3}


def build_library(force: bool = False) -> str:
    """Compiles gen.c into libgmwork.so with gcc and OpenMP."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O3", "-fopenmp", "-shared", "-fPIC", "-o", tmp, _SRC], check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _Csr(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int64), ("n_cols", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("row_ptr", ctypes.c_void_p), ("col", ctypes.c_void_p), ("val", ctypes.c_void_p)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build_library()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.POINTER(_Csr)
        lib.gm_gen_rmat.restype = P
        lib.gm_gen_rmat.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_double,
                                    ctypes.c_double, ctypes.c_uint64, ctypes.c_int32]
        lib.gm_gen_banded.restype = P
        lib.gm_gen_banded.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64, ctypes.c_int32]
        lib.gm_gen_erdos_renyi.restype = P
        lib.gm_gen_erdos_renyi.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64,
                                           ctypes.c_int32]
        lib.gm_gen_uniform.restype = P
        lib.gm_gen_uniform.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_double, ctypes.c_uint64,
                                       ctypes.c_int32]
        lib.gm_gen_free.argtypes = [P]
        lib.gm_gen_copy.argtypes = [P, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        lib.gm_gen_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


@dataclass
class CSR:
    """Canonical CSR matrix held in host numpy arrays."""

    n_rows: int
    n_cols: int
    row_ptr: np.ndarray  # int64, n_rows + 1
    col: np.ndarray  # int32 (int64 for column counts of 2^31 and more), nnz
    val: np.ndarray  # float64, nnz

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])

    def to_dense(self) -> np.ndarray:
        d = np.zeros((self.n_rows, self.n_cols), dtype=np.float64)
        rows = np.repeat(np.arange(self.n_rows), np.diff(self.row_ptr))
        d[rows, self.col] = self.val
        return d

    def pattern_dense(self) -> np.ndarray:
        d = np.zeros((self.n_rows, self.n_cols), dtype=bool)
        rows = np.repeat(np.arange(self.n_rows), np.diff(self.row_ptr))
        d[rows, self.col] = True
        return d

    def with_values(self, val: np.ndarray) -> "CSR":
        return CSR(self.n_rows, self.n_cols, self.row_ptr, self.col, np.ascontiguousarray(val, np.float64))


def _take(ptr) -> CSR:
    if not ptr:
        raise ValueError("generator rejected its arguments or ran out of memory")
    lib = _load()
    s = ptr.contents
    rp = np.empty(s.n_rows + 1, dtype=np.int64)
    col = np.empty(s.nnz, dtype=np.int32)
    val = np.empty(s.nnz, dtype=np.float64)
    lib.gm_gen_copy(ptr, rp.ctypes.data, col.ctypes.data, val.ctypes.data)
    out = CSR(int(s.n_rows), int(s.n_cols), rp, col, val)
    lib.gm_gen_free(ptr)
    return out


def rmat(scale: int, edge_factor: int, a: float, b: float, c: float, seed: int, values: str = "u01") -> CSR:
    """R-MAT: 2^scale square, edge_factor*2^scale quadrant draws, duplicates summed."""
    return _take(_load().gm_gen_rmat(scale, edge_factor, a, b, c, seed, VALUE_MODES[values]))


def banded(n: int, half: int, seed: int, values: str = "pm1") -> CSR:
    """Banded n x n with columns i-half..i+half clipped to [0, n)."""
    return _take(_load().gm_gen_banded(n, half, seed, VALUE_MODES[values]))


def erdos_renyi(n_rows: int, n_cols: int, d: int, seed: int, values: str = "pm1") -> CSR:
    """Exactly d distinct uniform columns per row."""
    return _take(_load().gm_gen_erdos_renyi(n_rows, n_cols, d, seed, VALUE_MODES[values]))


def uniform(n_rows: int, n_cols: int, density: float, seed: int, values: str = "pm1") -> CSR:
    """Every entry present independently with probability `density` (small sizes only)."""
    return _take(_load().gm_gen_uniform(n_rows, n_cols, density, seed, VALUE_MODES[values]))


def identity(n: int) -> CSR:
    return CSR(n, n, np.arange(n + 1, dtype=np.int64), np.arange(n, dtype=np.int32), np.ones(n))


def wide(n_rows: int, n_cols: int, per_row: int, seed: int, window: int = 0, base: int = -1) -> CSR:
    """CSR with int64 columns over a column range that may exceed 2^31: each
    row holds `per_row` distinct columns drawn uniformly (numpy's seeded
    generator) from the whole range, or, with window > 0, from a window of
    that many columns starting at `base` (placed at random per row when base
    is negative); values U(-1, 1)."""
    rng = np.random.default_rng(seed)
    cols = []
    for _ in range(n_rows):
        if window:
            lo = base if base >= 0 else int(rng.integers(0, max(n_cols - window, 1)))
            c = lo + rng.choice(min(window, n_cols), size=min(per_row, window), replace=False)
        else:
            c = rng.choice(n_cols, size=per_row, replace=False) if n_cols < (1 << 24) else \
                np.unique(rng.integers(0, n_cols, size=per_row))
        cols.append(np.sort(np.asarray(c, np.int64)))
    rp = np.zeros(n_rows + 1, np.int64)
    np.cumsum([c.size for c in cols], out=rp[1:])
    col = np.concatenate(cols) if cols else np.zeros(0, np.int64)
    return CSR(n_rows, n_cols, rp, col, rng.uniform(-1.0, 1.0, col.size))


def permutation(n: int, seed: int) -> CSR:
    """Permutation matrix P with P[i, perm[i]] = 1, perm drawn from a seeded numpy generator."""
    perm = np.random.default_rng(seed).permutation(n).astype(np.int32)
    return CSR(n, n, np.arange(n + 1, dtype=np.int64), perm, np.ones(n))


def empty(n_rows: int, n_cols: int) -> CSR:
    return CSR(n_rows, n_cols, np.zeros(n_rows + 1, np.int64), np.zeros(0, np.int32), np.zeros(0))


def generator_threads() -> int:
    return int(_load().gm_gen_threads())


@dataclass(frozen=True)
class Config:
    name: str
    kind: str
    params: tuple
    seed: int
    values: str

    def make(self) -> CSR:
        if self.kind == "rmat":
            scale, ef, a, b, c = self.params
            return rmat(scale, ef, a, b, c, self.seed, self.values)
        if self.kind == "banded":
            n, half = self.params
            return banded(n, half, self.seed, self.values)
        if self.kind == "er":
            n, d = self.params
            return erdos_renyi(n, n, d, self.seed, self.values)
        raise ValueError(self.kind)


@dataclass(frozen=True)
class PairConfig:
    """C = A*B with two R-MAT matrices of one scale and different densities
    (edge factors), Graph500 parameters a = 0.57, b = c = 0.19, as in the
    paper's RMat grid (Section IV-A)."""

    name: str
    scale: int
    a_edge_factor: int
    b_edge_factor: int
    seed: int

    def make(self) -> tuple:
        A = rmat(self.scale, self.a_edge_factor, 0.57, 0.19, 0.19, self.seed, "u01")
        B = rmat(self.scale, self.b_edge_factor, 0.57, 0.19, 0.19, self.seed + 1, "u01")
        return A, B


# A*B pairs of the RMat grid (A density 4..64, B density 4..16, scales 15..20).
PAIRS = {
    "rmat20_a32_b8": PairConfig("rmat20_a32_b8", 20, 32, 8, 2032),
    "rmat20_a64_b16": PairConfig("rmat20_a64_b16", 20, 64, 16, 2064),
}

# The five workloads, each multiplied by itself (C = A*A).
CONFIGS = {
    "rmat12": Config("rmat12", "rmat", (12, 8, 0.57, 0.19, 0.19), 12, "u01"),
    "banded20": Config("banded20", "banded", (1 << 20, 13), 20, "pm1"),
    "er22": Config("er22", "er", (1 << 22, 16), 22, "pm1"),
    "rmat22": Config("rmat22", "rmat", (22, 16, 0.57, 0.19, 0.19), 2222, "u01"),
    "rmat23": Config("rmat23", "rmat", (23, 8, 0.60, 0.17, 0.17), 2323, "u01"),
}
