"""CPU oracle for the gMAGNUS hot path (C = A*B on CSR).

TEST INFRASTRUCTURE ONLY. The test suite, the smoke check and the benchmark's
CPU-baseline leg may import this package; the GPU library and its Python
binding never do, and the two share no code. Inputs come from the separate
``workloads`` module, which holds no SpGEMM arithmetic.

Contents
--------
- :func:`spgemm` / :func:`row_products` -- plain Gustavson with a sorted,
  compensated per-row accumulator (C code in ``spgemm_oracle.c``; paper
  Section II-B, Eq. gustav and Algorithm 1).
- :func:`row_counts` -- the symbolic phase alone (distinct columns per row)
  by column marking, fast enough for whole R-MAT scale-22/23 products.
- :mod:`oracle.params` -- the parameter selection of Section III-D
  (``GetMagnusParams``), pinned to the chunk counts the paper prints.
- ``golden_structure.py`` -- writes the stored structure digests (nnz(C) and
  row-pointer hashes) of the large workloads from :func:`row_counts`.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "spgemm_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")


def build_library(force: bool = False) -> str:
    """Compiles the C oracle with gcc (-O2, OpenMP) into liboracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _Csr(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int64), ("n_cols", ctypes.c_int64), ("row_ptr", ctypes.c_void_p),
                ("col", ctypes.c_void_p), ("val", ctypes.c_void_p)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build_library()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.POINTER(_Csr)
        lib.oracle_row_products.argtypes = [P, P, ctypes.c_void_p]
        lib.oracle_count_rows.argtypes = [P, P, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_count_rows.restype = ctypes.c_int
        lib.oracle_fill_rows.argtypes = [P, P, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        lib.oracle_fill_rows.restype = ctypes.c_int
        lib.oracle_row_counts.argtypes = [P, P, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_row_counts.restype = ctypes.c_int
        lib.oracle_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _desc(m):
    rp = np.ascontiguousarray(m.row_ptr, np.int64)
    col = np.ascontiguousarray(m.col, np.int64)  # widened: the oracle reads 64-bit columns
    val = np.ascontiguousarray(m.val, np.float64)
    keep = (rp, col, val)
    return _Csr(m.n_rows, m.n_cols, rp.ctypes.data, col.ctypes.data, val.ctypes.data), keep


def _check_inner(A, B):
    if A.n_cols != B.n_rows:
        raise ValueError("inner dimensions differ: A is %dx%d, B is %dx%d" % (A.n_rows, A.n_cols, B.n_rows, B.n_cols))


def row_products(A, B) -> np.ndarray:
    """ip[i] = number of intermediate products of row i = sum_j nnz(B[A.col[j], :])."""
    _check_inner(A, B)
    da, ka = _desc(A)
    db, kb = _desc(B)
    ip = np.empty(A.n_rows, np.int64)
    _load().oracle_row_products(ctypes.byref(da), ctypes.byref(db), ip.ctypes.data)
    return ip


def row_counts(A, B, row_begin=0, row_end=None) -> np.ndarray:
    """Distinct columns of each row of C = A*B in [row_begin, row_end) (the
    symbolic phase, Section II-B), counted by marking columns; no products are
    formed, so whole R-MAT products take minutes on a few cores."""
    _check_inner(A, B)
    row_end = A.n_rows if row_end is None else row_end
    if not 0 <= row_begin <= row_end <= A.n_rows:
        raise ValueError("bad row range")
    da, ka = _desc(A)
    db, kb = _desc(B)
    counts = np.empty(row_end - row_begin, np.int64)
    if _load().oracle_row_counts(ctypes.byref(da), ctypes.byref(db), row_begin, row_end, counts.ctypes.data):
        raise MemoryError("oracle could not allocate its column stamps (or C has more than 2^31 columns)")
    return counts


@dataclass
class OracleRows:
    """Rows `rows` of C = A*B, packed as CSR in the order listed."""

    rows: np.ndarray  # int64 row ids
    row_ptr: np.ndarray  # int64, len(rows)+1
    col: np.ndarray  # int64
    val: np.ndarray  # float64
    bound: np.ndarray  # float64, sum |a*b| per entry
    terms: np.ndarray  # int64, products summed per entry

    def row(self, t):
        s, e = self.row_ptr[t], self.row_ptr[t + 1]
        return self.col[s:e], self.val[s:e], self.bound[s:e]

    def row_terms(self, t):
        return self.terms[self.row_ptr[t]:self.row_ptr[t + 1]]


def spgemm(A, B, rows=None) -> OracleRows:
    """Computes rows `rows` (default: all) of C = A*B, symbolic then numeric."""
    _check_inner(A, B)
    lib = _load()
    if rows is None:
        rows = np.arange(A.n_rows, dtype=np.int64)
    rows = np.ascontiguousarray(rows, np.int64)
    if rows.size and (rows.min() < 0 or rows.max() >= A.n_rows):
        raise ValueError("row index out of range")
    da, ka = _desc(A)
    db, kb = _desc(B)
    counts = np.empty(rows.size, np.int64)
    if lib.oracle_count_rows(ctypes.byref(da), ctypes.byref(db), rows.ctypes.data, rows.size, counts.ctypes.data):
        raise MemoryError("oracle could not expand a row")
    rp = np.zeros(rows.size + 1, np.int64)
    np.cumsum(counts, out=rp[1:])
    nnz = int(rp[-1])
    col = np.empty(nnz, np.int64)
    val = np.empty(nnz, np.float64)
    bound = np.empty(nnz, np.float64)
    terms = np.empty(nnz, np.int64)
    if lib.oracle_fill_rows(ctypes.byref(da), ctypes.byref(db), rows.ctypes.data, rows.size, rp.ctypes.data,
                            col.ctypes.data, val.ctypes.data, bound.ctypes.data, terms.ctypes.data):
        raise MemoryError("oracle could not expand a row")
    return OracleRows(rows, rp, col, val, bound, terms)


def threads() -> int:
    """OpenMP threads the oracle runs with."""
    return int(_load().oracle_threads())
