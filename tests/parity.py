"""Comparison of GPU results with the CPU oracle (shared by the GPU tests
and the smoke check).

The bar: row pointers and column indices identical; every value within
1e-12 * sum |a_ik * b_kj| of the oracle's (exact zero where that sum is 0).
"""
from __future__ import annotations

import numpy as np

import oracle

TOL = 1e-12


def compare_rows(rows, gpu_rp, gpu_col, gpu_val, ref: "oracle.OracleRows"):
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
        err = np.abs(gpu_val[s:e] - v_ref)
        lim = TOL * b_ref
        if np.any(err > lim):
            bad = int(np.nonzero(err > lim)[0][0])
            raise AssertionError("row %d col %d: value %r, oracle %r, bound %r" % (i, c[bad], gpu_val[s + bad],
                                                                                   v_ref[bad], b_ref[bad]))
        with np.errstate(divide="ignore", invalid="ignore"):
            r = np.where(b_ref > 0, err / b_ref, 0.0)
        if r.size:
            worst = max(worst, float(r.max()))
    return worst


def compare_full(gpu_rp, gpu_col, gpu_val, ref: "oracle.OracleRows"):
    """Whole matrix: row pointers bit-exact, then every row."""
    if not np.array_equal(gpu_rp, ref.row_ptr):
        bad = int(np.nonzero(gpu_rp != ref.row_ptr)[0][0])
        raise AssertionError("row_ptr differs first at %d: %d vs oracle %d" % (bad, gpu_rp[bad], ref.row_ptr[bad]))
    if not np.array_equal(gpu_col, ref.col):
        bad = int(np.nonzero(gpu_col != ref.col)[0][0])
        raise AssertionError("col differs first at %d" % bad)
    err = np.abs(gpu_val - ref.val)
    lim = TOL * ref.bound
    if np.any(err > lim):
        bad = int(np.nonzero(err > lim)[0][0])
        raise AssertionError("value %d: %r vs oracle %r (bound %r)" % (bad, gpu_val[bad], ref.val[bad], ref.bound[bad]))
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(ref.bound > 0, err / ref.bound, 0.0)
    return float(r.max()) if r.size else 0.0
