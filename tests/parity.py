"""Comparison of GPU results with the CPU oracle (shared by the GPU tests
and the smoke check).

The bar: row pointers and column indices identical; every value within
1e-12 * sum |a_ik * b_kj| of the oracle's (exact zero where that sum is 0).
For fp32 values the bar is (n + 1) * 2^-24 * sum |a_ik * b_kj| with n the
entry's number of products: every product and each of the n - 1 additions,
in any order, round once with relative error at most 2^-24, so the first-
order worst case of the summation is n * 2^-24 * sum |ab|; the oracle's own
value (fp32 inputs widened, exact fp64 products, compensated sum) is exact
to about one fp64 rounding.
"""
from __future__ import annotations

import numpy as np

import oracle

TOL = 1e-12
U32 = 2.0 ** -24


def tolerance(bound, terms, f32: bool):
    """Per-entry bound on |c - c_ref|."""
    return (terms + 1.0) * U32 * bound if f32 else TOL * bound


def compare_rows(rows, gpu_rp, gpu_col, gpu_val, ref: "oracle.OracleRows", f32: bool = False):
    """rows: row ids (into gpu_rp). Returns the max relative error; raises on mismatch."""
    worst = 0.0
    for t, i in enumerate(rows):
        s, e = int(gpu_rp[i]), int(gpu_rp[i + 1])
        c_ref, v_ref, b_ref = ref.row(t)
        if e - s != c_ref.size:
            raise AssertionError("row %d: %d entries, oracle has %d" % (i, e - s, c_ref.size))
        c = gpu_col[s:e]
        if not np.array_equal(c, c_ref):
            bad = int(np.nonzero(c != c_ref)[0][0])
            raise AssertionError("row %d: column %d is %d, oracle %d" % (i, bad, c[bad], c_ref[bad]))
        err = np.abs(gpu_val[s:e].astype(np.float64) - v_ref)
        lim = tolerance(b_ref, ref.row_terms(t), f32)
        if np.any(err > lim):
            bad = int(np.nonzero(err > lim)[0][0])
            raise AssertionError("row %d col %d: value %r, oracle %r, bound %r" % (i, c[bad], gpu_val[s + bad],
                                                                                   v_ref[bad], b_ref[bad]))
        with np.errstate(divide="ignore", invalid="ignore"):
            r = np.where(b_ref > 0, err / b_ref, 0.0)
        if r.size:
            worst = max(worst, float(r.max()))
    return worst


def compare_full(gpu_rp, gpu_col, gpu_val, ref: "oracle.OracleRows", f32: bool = False):
    """Whole matrix: row pointers bit-exact, then every row."""
    if not np.array_equal(gpu_rp, ref.row_ptr):
        bad = int(np.nonzero(gpu_rp != ref.row_ptr)[0][0])
        raise AssertionError("row_ptr differs first at %d: %d vs oracle %d" % (bad, gpu_rp[bad], ref.row_ptr[bad]))
    if not np.array_equal(gpu_col, ref.col):
        bad = int(np.nonzero(gpu_col != ref.col)[0][0])
        raise AssertionError("col differs first at %d" % bad)
    err = np.abs(gpu_val.astype(np.float64) - ref.val)
    lim = tolerance(ref.bound, ref.terms, f32)
    if np.any(err > lim):
        bad = int(np.nonzero(err > lim)[0][0])
        raise AssertionError("value %d: %r vs oracle %r (bound %r)" % (bad, gpu_val[bad], ref.val[bad], ref.bound[bad]))
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(ref.bound > 0, err / ref.bound, 0.0)
    return float(r.max()) if r.size else 0.0
