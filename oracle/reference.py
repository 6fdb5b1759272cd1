"""Small numpy references for the heavy-row reorder steps (toy sizes only).

TEST INFRASTRUCTURE ONLY (see the package docstring).

- :func:`split_rows` -- the light/heavy split of rows by intermediate-product
  count (Algorithm 3, ThreshPartition: heavy iff ip > tau).
- :func:`expand` -- the intermediate matrix C-hat of the heavy rows
  (Section III-B, Eq. outer): row h of C-hat holds every product
  A[x_heavy[h], k] * B[k, j] as a (j, value) pair, in no particular order,
  so it is returned as a multiset (sorted by column, then value).
- :func:`multisplit` -- one level of the range multisplit (Section III-C):
  row r of the input is cut into n_chunks column ranges of width
  m_out = m_in / n_chunks; chunk (r, c) keeps the pairs with
  column // m_out == c, with the column shifted to column - c*m_out
  (Section III-A: the shift into the local chunk range, undone on the final
  write). Chunks above tau are listed first, each group in (r, c) order, the
  order that lets the next level read the heavy chunks contiguously.
"""
from __future__ import annotations

import numpy as np


def split_rows(ip: np.ndarray, tau: int):
    ip = np.asarray(ip)
    heavy = np.nonzero(ip > tau)[0].astype(np.int64)
    light = np.nonzero(ip <= tau)[0].astype(np.int64)
    return heavy, light


def _canon(cols, vals):
    cols = np.asarray(cols, np.int64)
    vals = np.asarray(vals, np.float64)
    order = np.lexsort((vals, cols))
    return cols[order], vals[order]


def expand(A, B, rows):
    """List over `rows` of (cols, vals) multisets of each row's products."""
    out = []
    for i in rows:
        cs, vs = [], []
        for p in range(A.row_ptr[i], A.row_ptr[i + 1]):
            k = A.col[p]
            s, e = B.row_ptr[k], B.row_ptr[k + 1]
            cs.append(B.col[s:e])
            vs.append(A.val[p] * B.val[s:e])
        if cs:
            out.append(_canon(np.concatenate(cs), np.concatenate(vs)))
        else:
            out.append((np.zeros(0, np.int64), np.zeros(0)))
    return out


def multisplit(rows, m_in: int, n_chunks: int, tau: int | None = None):
    """One level: returns (chunks, order, heavy_count).

    chunks[(r, c)] = (cols shifted into [0, m_out), vals) as a multiset.
    order lists the (r, c) keys heavy first (count > tau), then light; with
    tau None every chunk counts as light (the last level).
    """
    if m_in % n_chunks:
        raise ValueError("chunk count must divide the column range")
    m_out = m_in // n_chunks
    chunks = {}
    for r, (cols, vals) in enumerate(rows):
        cols = np.asarray(cols, np.int64)
        if cols.size and (cols.min() < 0 or cols.max() >= m_in):
            raise ValueError("column outside the row's range")
        which = cols // m_out
        for c in range(n_chunks):
            sel = which == c
            chunks[(r, c)] = _canon(cols[sel] - c * m_out, np.asarray(vals)[sel])
    keys = [(r, c) for r in range(len(rows)) for c in range(n_chunks)]
    heavy = [k for k in keys if tau is not None and chunks[k][0].size > tau]
    light = [k for k in keys if not (tau is not None and chunks[k][0].size > tau)]
    return chunks, heavy + light, len(heavy)
