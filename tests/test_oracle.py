"""Pins of the CPU oracle against facts fixed by the paper or by mathematics.

Each pin is independent of the oracle's own algorithm (gather, stable sort,
compensated run reduction): dense products from numpy, closed forms counted
by hand, exact integer arithmetic, identities, and brute force on tiny
inputs. A plausible mistake in the oracle (a dropped product, a wrong index,
a transposed operand, lost structural zeros, uncompensated sums) fails at
least one of them.
"""
import os

import numpy as np
import pytest

import oracle
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def full(A, B):
    return oracle.spgemm(A, B)


def as_csr(r: oracle.OracleRows, n_cols):
    return wl.CSR(len(r.rows), n_cols, r.row_ptr, r.col, r.val)


def csr_transpose_dense_check(C, dense):
    got = as_csr(C, dense.shape[1]).to_dense()
    return got


SHAPES = [(1, 1, 1), (5, 7, 3), (17, 40, 23), (64, 64, 64), (33, 9, 50), (0, 4, 4), (6, 0, 5)]


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("density", [0.0, 0.05, 0.3, 0.8])
def test_dense_bruteforce(shape, density):
    m, k, n = shape
    seed = hash((shape, density)) & 0xFFFF
    A = wl.uniform(m, max(k, 1), density, seed) if k else wl.empty(m, 0)
    B = wl.uniform(k, n, density, seed + 1) if k else wl.empty(0, n)
    if k == 0:
        A = wl.CSR(m, 0, np.zeros(m + 1, np.int64), np.zeros(0, np.int32), np.zeros(0))
    C = full(A, B)
    # structure: boolean product of the patterns
    pa = A.pattern_dense().astype(np.int64) if k else np.zeros((m, 0), np.int64)
    pb = B.pattern_dense().astype(np.int64)
    pattern = (pa @ pb) > 0
    got = as_csr(C, n)
    assert np.array_equal(got.pattern_dense(), pattern)
    # columns strictly increasing within each row
    for t in range(m):
        c = C.col[C.row_ptr[t]:C.row_ptr[t + 1]]
        assert np.all(np.diff(c) > 0)
    # values: dense fp64 product, within a tight multiple of the bound
    dense = (A.to_dense() if k else np.zeros((m, 0))) @ B.to_dense()
    rows = np.repeat(np.arange(m), np.diff(C.row_ptr))
    ref = dense[rows, C.col]
    assert np.all(np.abs(C.val - ref) <= 1e-14 * C.bound + 1e-300)
    # bound = sum of |a*b| = |A| @ |B|
    absd = (np.abs(A.to_dense()) if k else np.zeros((m, 0))) @ np.abs(B.to_dense())
    assert np.allclose(C.bound, absd[rows, C.col], rtol=1e-14, atol=0)
    # terms = number of products per entry = the integer product of the patterns
    counts = pa @ pb
    assert np.array_equal(C.terms, counts[rows, C.col])


def test_identity_and_permutation_exact():
    A = wl.rmat(9, 8, 0.57, 0.19, 0.19, 5)
    n = A.n_rows
    I = wl.identity(n)
    for C in (full(I, A), full(A, I)):
        assert np.array_equal(C.row_ptr, A.row_ptr)
        assert np.array_equal(C.col, A.col)
        assert np.array_equal(C.val, A.val)  # one product per entry: bit-exact
    P = wl.permutation(n, 3)
    perm = P.col.astype(np.int64)  # P[i, perm[i]] = 1
    # (P A)[i, :] = A[perm[i], :]
    PA = full(P, A)
    for i in range(0, n, 7):
        s, e = A.row_ptr[perm[i]], A.row_ptr[perm[i] + 1]
        c, v, _ = PA.row(i)
        assert np.array_equal(c, A.col[s:e]) and np.array_equal(v, A.val[s:e])
    # (A P)[i, perm[j]] = A[i, j]
    AP = full(A, P)
    for i in range(0, n, 5):
        s, e = A.row_ptr[i], A.row_ptr[i + 1]
        cols = perm[A.col[s:e]]
        order = np.argsort(cols)
        c, v, _ = AP.row(i)
        assert np.array_equal(c, cols[order]) and np.array_equal(v, A.val[s:e][order])


def test_integer_values_exact():
    # every partial sum of small integers is exact in fp64, in any order
    A = wl.uniform(48, 60, 0.3, 11, values="int3")
    B = wl.uniform(60, 52, 0.3, 12, values="int3")
    C = full(A, B)
    dense = A.to_dense().astype(np.int64) @ B.to_dense().astype(np.int64)
    rows = np.repeat(np.arange(48), np.diff(C.row_ptr))
    assert np.array_equal(C.val, dense[rows, C.col].astype(np.float64))
    # integer-valued R-MAT: sampled rows against exact per-row integer sums
    R = wl.rmat(10, 8, 0.57, 0.19, 0.19, 4, values="int3")
    CR = oracle.spgemm(R, R, rows=np.arange(0, R.n_rows, 3))
    for t, i in enumerate(CR.rows):
        acc = {}
        for p in range(R.row_ptr[i], R.row_ptr[i + 1]):
            k = R.col[p]
            for q in range(R.row_ptr[k], R.row_ptr[k + 1]):
                acc[int(R.col[q])] = acc.get(int(R.col[q]), 0) + int(R.val[p]) * int(R.val[q])
        c, v, _ = CR.row(t)
        assert list(c) == sorted(acc)
        assert np.array_equal(v, np.array([acc[j] for j in sorted(acc)], np.float64))


def _golden_rows(name):
    out = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                out.append([x.strip() for x in line.split("|")])
    return out


@pytest.mark.parametrize("n", [200, 4096])
def test_banded_closed_forms(n):
    row = [r for r in _golden_rows("banded_closed_forms.txt") if int(r[0]) == n][0]
    A = wl.banded(n, 13, 1, values="ones")
    assert A.nnz == int(row[1])
    ip = oracle.row_products(A, A)
    assert int(ip.sum()) == int(row[2])
    C = full(A, A)
    assert int(C.row_ptr[-1]) == int(row[3])
    # value of every entry: number of k within 13 of both i and j (brute force)
    rows = np.repeat(np.arange(n), np.diff(C.row_ptr))
    ks = np.arange(n)
    sample = np.arange(0, C.col.size, max(1, C.col.size // 3000))
    for e in sample:
        i, j = rows[e], C.col[e]
        cnt = np.count_nonzero((np.abs(ks - i) <= 13) & (np.abs(ks - j) <= 13))
        assert C.val[e] == cnt
        if 26 <= i < n - 26:
            assert C.val[e] == 27 - abs(int(i) - int(j))


def test_banded_full_size_counts():
    row = [r for r in _golden_rows("banded_closed_forms.txt") if int(r[0]) == 1 << 20][0]
    A = wl.CONFIGS["banded20"].make()
    assert A.nnz == int(row[1])
    assert int(oracle.row_products(A, A).sum()) == int(row[2])


def test_er_products_per_row():
    A = wl.erdos_renyi(4096, 4096, 16, 9)
    assert np.all(np.diff(A.row_ptr) == 16)
    assert np.all(oracle.row_products(A, A) == 256)


@pytest.mark.parametrize("seed", [1, 2])
def test_product_count_invariant(seed):
    A = wl.rmat(11, 8, 0.57, 0.19, 0.19, seed)
    B = wl.rmat(11, 4, 0.57, 0.19, 0.19, seed + 10)
    ip = oracle.row_products(A, B)
    colcount = np.bincount(A.col, minlength=A.n_cols)
    rowlen = np.diff(B.row_ptr)
    assert int(ip.sum()) == int((colcount * rowlen).sum())
    # symbolic counts never exceed the product counts, and equal the distinct count
    C = full(A, B)
    assert np.all(np.diff(C.row_ptr) <= ip)


def test_compensated_reduction():
    # products 1e16, 1, -1e16 on one column: plain left-to-right summation gives 0
    A = wl.CSR(1, 3, np.array([0, 3], np.int64), np.array([0, 1, 2], np.int32), np.array([1e16, 1.0, -1e16]))
    B = wl.CSR(3, 2, np.array([0, 1, 2, 3], np.int64), np.array([1, 1, 1], np.int32), np.ones(3))
    C = full(A, B)
    assert list(C.col) == [1]
    assert C.val[0] == 1.0
    assert C.bound[0] == 2e16 + 1.0


def test_structural_zero_kept():
    # products +2 and -2 cancel exactly; the entry stays with value 0
    A = wl.CSR(1, 2, np.array([0, 2], np.int64), np.array([0, 1], np.int32), np.array([1.0, -1.0]))
    B = wl.CSR(2, 3, np.array([0, 2, 3], np.int64), np.array([0, 2, 2], np.int32), np.array([5.0, 2.0, 2.0]))
    C = full(A, B)
    assert list(C.col) == [0, 2]
    assert list(C.val) == [5.0, 0.0]


def test_rows_subset_matches_full():
    A = wl.rmat(10, 8, 0.57, 0.19, 0.19, 8)
    F = full(A, A)
    rows = np.array([0, 5, 1023, 17, 5])
    S = oracle.spgemm(A, A, rows=rows)
    for t, i in enumerate(rows):
        c, v, b = S.row(t)
        s, e = F.row_ptr[i], F.row_ptr[i + 1]
        assert np.array_equal(c, F.col[s:e]) and np.array_equal(v, F.val[s:e])


def test_rejects_mismatched_shapes():
    A = wl.uniform(4, 5, 0.5, 1)
    with pytest.raises(ValueError):
        oracle.spgemm(A, A)


def test_rmat_generator_against_paper_table():
    # Table "Properties of the representative RMat matrices": scale 15,
    # B density 8; C.nnz / C.n = 477.6 (A density 4) and 782.3 (A density 8).
    B = wl.rmat(15, 8, 0.57, 0.19, 0.19, 101)
    for dens, printed in ((4, 477.6), (8, 782.3)):
        A = wl.rmat(15, dens, 0.57, 0.19, 0.19, 200 + dens)
        C = full(A, B)
        ratio = C.row_ptr[-1] / A.n_rows
        assert abs(ratio - printed) <= 0.15 * printed, (dens, ratio, printed)


def test_rmat12_workload_shape():
    A = wl.CONFIGS["rmat12"].make()
    assert A.n_rows == 4096 and 27000 < A.nnz < 30000
    rl = np.diff(A.row_ptr)
    for i in range(A.n_rows):
        c = A.col[A.row_ptr[i]:A.row_ptr[i + 1]]
        assert np.all(np.diff(c) > 0)
    assert rl.sum() == A.nnz and np.all(A.val > 0)


# ---------------------------------------------------------------- planner pins

def _parse_table(s):
    s = s.strip()
    if s == "N/A":
        return None
    if ":" in s:
        req, rest = s.split(":")
        return int(req), [int(x) for x in rest.split(",")]
    return int(s), [int(s)]


def test_planner_reproduces_printed_chunk_counts():
    from oracle.params import get_magnus_params

    n_checked = 0
    for name, cm, pvc, h200 in _golden_rows("num_chunks.txt"):
        for s_lm, printed in ((131072, pvc), (233472, h200)):
            exp = _parse_table(printed)
            if exp is None:
                continue
            p = get_magnus_params(int(cm), s_lm)
            assert (p.chunks_required, p.v_chunks) == exp, (name, s_lm, p)
            assert p.table_string() == printed.strip()
            n_checked += 1
    assert n_checked == 51


def test_planner_mi355x_values():
    from oracle.params import get_magnus_params

    p = get_magnus_params(1 << 22, 163840)
    assert (p.tau, p.dense_width, p.chunks_max, p.group_rows) == (6826, 8192, 32, 2)
    assert p.v_chunks == [32, 16]
    assert get_magnus_params(1 << 23, 163840).v_chunks == [32, 32]
    assert get_magnus_params(4096, 163840).v_chunks == []
    # paper: n_groupRows = 2 in its experiments
    assert get_magnus_params(1 << 20, 131072).group_rows == 2
    assert get_magnus_params(1 << 20, 233472).group_rows == 2


# ------------------------------------------------------ 64-bit column indices

def test_wide_columns_bruteforce():
    # B with columns spread over 2^33: each row of C accumulated in a Python
    # dict from the definition (Section II-B, Eq. gustav), compared entry by
    # entry (columns exact, values within a few roundings, term counts exact)
    A = wl.uniform(25, 30, 0.2, 41)
    for B in (wl.wide(30, 1 << 33, 6, 42), wl.wide(30, 1 << 33, 9, 43, window=40)):
        C = oracle.spgemm(A, B)
        for i in range(A.n_rows):
            acc, mag, cnt = {}, {}, {}
            for p in range(A.row_ptr[i], A.row_ptr[i + 1]):
                k = int(A.col[p])
                for r in range(B.row_ptr[k], B.row_ptr[k + 1]):
                    c = int(B.col[r])
                    x = float(A.val[p]) * float(B.val[r])
                    acc[c] = acc.get(c, 0.0) + x
                    mag[c] = mag.get(c, 0.0) + abs(x)
                    cnt[c] = cnt.get(c, 0) + 1
            cols = sorted(acc)
            c_ref, v_ref, b_ref = C.row(i)
            assert list(c_ref) == cols
            assert np.allclose(v_ref, [acc[c] for c in cols], rtol=0, atol=1e-14 * max(mag.values(), default=1))
            assert list(C.row_terms(i)) == [cnt[c] for c in cols]


def test_column_shift_moves_columns_only():
    # shifting every column of B by 2^32 shifts the columns of C by 2^32 and
    # leaves values, bounds and term counts unchanged
    A = wl.rmat(8, 8, 0.57, 0.19, 0.19, 44)
    C = oracle.spgemm(A, A)
    B2 = wl.CSR(A.n_rows, A.n_cols + (1 << 32), A.row_ptr, A.col.astype(np.int64) + (1 << 32), A.val)
    C2 = oracle.spgemm(A, B2)
    assert np.array_equal(C2.row_ptr, C.row_ptr) and np.array_equal(C2.col, C.col + (1 << 32))
    assert np.array_equal(C2.val, C.val) and np.array_equal(C2.bound, C.bound)
    assert np.array_equal(C2.terms, C.terms)


def test_terms_sum_to_row_products():
    A = wl.rmat(10, 8, 0.57, 0.19, 0.19, 45)
    C = oracle.spgemm(A, A)
    ip = oracle.row_products(A, A)
    cs = np.concatenate([[0], np.cumsum(C.terms)])
    assert np.array_equal(cs[C.row_ptr[1:]] - cs[C.row_ptr[:-1]], ip)


# ------------------------------------------------- symbolic counts by marking

@pytest.mark.parametrize("make", [
    lambda: (wl.rmat(11, 8, 0.57, 0.19, 0.19, 7),) * 2,
    lambda: (wl.uniform(300, 200, 0.05, 8), wl.uniform(200, 500, 0.03, 9)),
    lambda: (wl.banded(3000, 13, 10),) * 2,
    lambda: (wl.erdos_renyi(2000, 2000, 16, 11),) * 2,
    lambda: (wl.empty(7, 5), wl.uniform(5, 9, 0.5, 12)),
])
def test_row_counts_match_sorted_runs(make):
    # two independent ways to the symbolic result: runs of the stably sorted
    # products (spgemm) and column marking without any product (row_counts)
    A, B = make()
    C = oracle.spgemm(A, B)
    counts = oracle.row_counts(A, B)
    assert np.array_equal(counts, np.diff(C.row_ptr))
    # a row range gives the same counts as the whole
    a, b = A.n_rows // 3, A.n_rows - A.n_rows // 4
    assert np.array_equal(oracle.row_counts(A, B, a, b), counts[a:b])


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_row_counts_dense_pattern(seed):
    A = wl.uniform(40, 30, 0.15, seed)
    B = wl.uniform(30, 50, 0.1, seed + 10)
    pattern = (A.pattern_dense().astype(np.int64) @ B.pattern_dense().astype(np.int64)) > 0
    assert np.array_equal(oracle.row_counts(A, B), pattern.sum(axis=1))


def test_row_counts_banded_closed_form():
    # half-width 13: row i of C spans columns max(0, i-26) .. min(n-1, i+26)
    n = 1 << 16
    A = wl.banded(n, 13, 3)
    counts = oracle.row_counts(A, A)
    i = np.arange(n)
    assert np.array_equal(counts, np.minimum(n - 1, i + 26) - np.maximum(0, i - 26) + 1)
    assert int(counts.sum()) == 53 * n - 702


def test_structure_golden_files():
    # the stored digests of the full-size workloads are internally consistent
    # and agree with the closed forms where one exists
    from oracle import golden_structure

    for name in golden_structure.DEFAULT:
        g = golden_structure.read(name)
        assert g["config"] == name and len(g["blocks"]) == g["n_blocks"]
        assert sum(b[2] for b in g["blocks"]) == g["nnz_c"]
        assert g["blocks"][0][0] == 0 and g["blocks"][-1][1] == g["n_rows"]
        assert all(x[1] == y[0] for x, y in zip(g["blocks"][:-1], g["blocks"][1:]))
    b = golden_structure.read("banded20")
    n = b["n_rows"]
    assert b["nnz_c"] == 53 * n - 702 and b["products"] == 729 * n - 8190 and b["nnz_a"] == 27 * n - 182
    e = golden_structure.read("er22")
    assert e["products"] == 1 << 30 and (1 << 30) - 100_000 < e["nnz_c"] <= 1 << 30


def test_structure_digests_small():
    # the digest of a small matrix's counts, recomputed from its row pointers
    import hashlib

    from oracle import golden_structure

    A = wl.rmat(10, 8, 0.57, 0.19, 0.19, 4)
    C = oracle.spgemm(A, A)
    whole, per = golden_structure.structure_digests(oracle.row_counts(A, A), 8)
    assert whole == hashlib.sha256(np.ascontiguousarray(C.row_ptr, "<i8").tobytes()).hexdigest()
    assert sum(p[2] for p in per) == C.row_ptr[-1]
