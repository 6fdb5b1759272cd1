"""Parity at the five benchmark workloads' full sizes (and one R-MAT A*B pair),
in the benchmark's launch configuration (row panels of at most 4e9 products).

The whole product runs on the GPU, panel by panel. For every workload whose
C is too large to hold twice in host memory, the check has three parts:

- structure of the whole C: every row's count against the oracle's symbolic
  phase, through the stored digests under tests/golden/ (nnz(C), sha256 of
  the whole row-pointer array, and per block of rows); the digests were
  written by oracle/golden_structure.py, which calls only the oracle;
- one contiguous slice of rows, from row 0 until it holds at least 1e9
  products (the R-MAT hub rows sit at the lowest indices), compared entry by
  entry with the oracle: columns exact, values within the tolerance;
- randomly sampled rows, compared the same way.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from oracle import golden_structure
from tests.parity import compare_rows

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

PANEL_PRODUCTS = 4_000_000_000
SLICE_PRODUCTS = 1_000_000_000


@pytest.fixture(scope="module")
def g():
    from paper_2607_22866_amd import gmagnus

    gmagnus.load()
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return gmagnus


def sample_rows(ip, n_random, n_heaviest, seed):
    rng = np.random.default_rng(seed)
    rows = set(rng.choice(ip.size, size=min(n_random, ip.size), replace=False).tolist())
    rows.update(np.argsort(ip)[-n_heaviest:].tolist())
    rows.update([0, ip.size - 1])
    return np.array(sorted(rows), dtype=np.int64)


def leading_slice(ip, products):
    """Rows [0, r) with r the first row count whose products reach `products` (all rows if fewer)."""
    pre = np.cumsum(ip)
    r = int(np.searchsorted(pre, products)) + 1
    return np.arange(min(r, ip.size), dtype=np.int64)


def run_full(g, A, rows, panel_products=PANEL_PRODUCTS, B=None, new_values=None):
    """Runs C = A*A (A*B when B is given) panel by panel. Returns the row
    counts of every row of C, the listed rows' CSR and the totals. With
    new_values = (a_val, b_val) every panel's plan keeps its pattern, and C is
    recomputed for those values after the first numeric phase (the listed rows
    are those of the second result)."""
    dA = g.DeviceCSR.from_host(A)
    dB = dA if B is None else g.DeviceCSR.from_host(B)
    bounds = g.split_panels(dA, dB, panel_products)
    if new_values is not None:
        va = torch.from_numpy(new_values[0]).cuda()
        vb = va if B is None else torch.from_numpy(new_values[1]).cuda()
    counts = np.empty(A.n_rows, np.int64)
    out_rp = [0]
    out_col, out_val = [], []
    total_nnz = total_products = 0
    for a, b in zip(bounds[:-1], bounds[1:]):
        sel = rows[(rows >= a) & (rows < b)]
        with g.Plan(dA, dB, row_begin=a, row_end=b, flags=0 if new_values is None else g.FLAG_KEEP_PATTERN) as p:
            rp, nnz = p.symbolic()
            col, val = p.numeric()
            if new_values is not None:
                p.update_values(va, vb)
                p.numeric(col, val)
            info = p.info()
        assert info.check_flags == 0
        total_nnz += nnz
        total_products += info.products_total
        rp_h = rp.cpu().numpy()
        counts[a:b] = np.diff(rp_h)
        # one copy per run of consecutive listed rows
        runs = np.split(sel, np.nonzero(np.diff(sel) != 1)[0] + 1) if sel.size else []
        for run in runs:
            s0, e0 = int(rp_h[run[0] - a]), int(rp_h[run[-1] - a + 1])
            out_col.append(col[s0:e0].cpu().numpy())
            out_val.append(val[s0:e0].cpu().numpy())
            out_rp.extend((out_rp[-1] + rp_h[run + 1 - a] - s0).tolist())
        del rp, col, val
    torch.cuda.synchronize()
    return (counts, np.array(out_rp, np.int64), np.concatenate(out_col) if out_col else np.zeros(0, np.int32),
            np.concatenate(out_val) if out_val else np.zeros(0), total_nnz, total_products, len(bounds) - 1)


def check_structure(name, counts):
    """Every row count against the stored oracle digests."""
    ref = golden_structure.read(name)
    assert counts.size == ref["n_rows"]
    whole, per = golden_structure.structure_digests(counts, len(ref["blocks"]))
    bad = [(r, m) for r, m in zip(ref["blocks"], per) if r != m]
    if bad:
        (s, e, nz, _), (_, _, nz_gpu, _) = bad[0]
        raise AssertionError("%s: %d of %d row blocks differ from the oracle; first rows %d..%d: nnz %d, oracle %d" % (
            name, len(bad), len(per), s, e, nz_gpu, nz))
    assert int(counts.sum()) == ref["nnz_c"]
    assert whole == ref["row_ptr_sha256"]
    return ref


def check_config(g, name, n_random, n_heaviest, slice_products=0):
    A = wl.CONFIGS[name].make()
    ip = oracle.row_products(A, A)
    rows = sample_rows(ip, n_random, n_heaviest, seed=len(name))
    if slice_products:
        rows = np.union1d(rows, leading_slice(ip, slice_products))
    counts, rp, col, val, nnz, products, panels = run_full(g, A, rows)
    assert products == int(ip.sum())
    ref = check_structure(name, counts)
    assert ref["products"] == products and nnz == ref["nnz_c"]
    worst = compare_rows(np.arange(rows.size), rp, col, val, oracle.spgemm(A, A, rows=rows))
    print("%s: panels=%d products=%d nnz(C)=%d (all row counts match the oracle) rows compared=%d "
          "(products %d) max_rel_err=%.2e" % (name, panels, products, nnz, rows.size, int(ip[rows].sum()), worst))
    return A, ip, nnz


def test_banded20_full(g):
    A, ip, nnz = check_config(g, "banded20", 3000, 5)
    n = A.n_rows
    assert A.nnz == 27 * n - 182 and int(ip.sum()) == 729 * n - 8190 and nnz == 53 * n - 702


def test_er22_full(g):
    A, ip, nnz = check_config(g, "er22", 3000, 5)
    assert int(ip.sum()) == 1 << 30 and np.all(ip == 256)


def test_rmat22_full(g):
    check_config(g, "rmat22", 400, 3, SLICE_PRODUCTS)


def test_rmat23_full(g):
    check_config(g, "rmat23", 400, 3, SLICE_PRODUCTS)


def test_rmat20_pair_full(g):
    # C = A*B, R-MAT scale 20 with A edge factor 32 and B edge factor 8
    A, B = wl.PAIRS["rmat20_a32_b8"].make()
    ip = oracle.row_products(A, B)
    rows = sample_rows(ip, 400, 3, seed=20)
    counts, rp, col, val, nnz, products, panels = run_full(g, A, rows, B=B)
    assert products == int(ip.sum())
    assert np.array_equal(counts, oracle.row_counts(A, B))
    ref = oracle.spgemm(A, B, rows=rows)
    worst = compare_rows(np.arange(rows.size), rp, col, val, ref)
    print("rmat20_a32_b8: panels=%d products=%d nnz(C)=%d (all row counts match the oracle) sampled_rows=%d "
          "max_rel_err=%.2e" % (panels, products, nnz, rows.size, worst))


def test_rmat20_pair_pattern_reuse_full(g):
    # the same pair at full size, every panel recomputed for new values of A
    # and B on its kept pattern; sampled rows against the oracle's for the new values
    A, B = wl.PAIRS["rmat20_a32_b8"].make()
    rng = np.random.default_rng(21)
    A2 = A.with_values(rng.uniform(-1.0, 1.0, A.nnz))
    B2 = B.with_values(rng.uniform(-1.0, 1.0, B.nnz))
    ip = oracle.row_products(A, B)
    rows = sample_rows(ip, 300, 3, seed=21)
    counts, rp, col, val, nnz, products, panels = run_full(g, A, rows, B=B, new_values=(A2.val, B2.val))
    assert products == int(ip.sum())
    worst = compare_rows(np.arange(rows.size), rp, col, val, oracle.spgemm(A2, B2, rows=rows))
    print("rmat20_a32_b8 new values: panels=%d nnz(C)=%d sampled_rows=%d max_rel_err=%.2e" % (
        panels, nnz, rows.size, worst))
