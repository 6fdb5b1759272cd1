"""Parity at the five benchmark workloads' full sizes (and one R-MAT A*B pair), in the benchmark's
launch configuration (row panels of at most 4e9 products): the whole product
runs on the GPU, and sampled rows (random rows plus the heaviest rows) are
compared with the oracle, which computes them one by one. Properties that
hold at any size are checked on all rows: product totals against the
oracle's row counts, and the banded closed forms."""
import numpy as np
import pytest

import oracle
import workloads as wl
from tests.parity import compare_rows

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

PANEL_PRODUCTS = 4_000_000_000


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


def run_sampled(g, A, rows, panel_products=PANEL_PRODUCTS, B=None, new_values=None):
    """Runs C = A*A (A*B when B is given) panel by panel; returns the sampled
    rows' CSR and totals. With new_values = (a_val, b_val) every panel's plan
    keeps its pattern, and C is recomputed for those values after the first
    numeric phase (the sampled rows are those of the second result)."""
    dA = g.DeviceCSR.from_host(A)
    dB = dA if B is None else g.DeviceCSR.from_host(B)
    bounds = g.split_panels(dA, dB, panel_products)
    if new_values is not None:
        va = torch.from_numpy(new_values[0]).cuda()
        vb = va if B is None else torch.from_numpy(new_values[1]).cuda()
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
        if sel.size:
            rp_h = rp.cpu().numpy()
            for r in sel:
                s, e = int(rp_h[r - a]), int(rp_h[r - a + 1])
                out_col.append(col[s:e].cpu().numpy())
                out_val.append(val[s:e].cpu().numpy())
                out_rp.append(out_rp[-1] + e - s)
        del rp, col, val
    torch.cuda.synchronize()
    return (np.array(out_rp, np.int64), np.concatenate(out_col) if out_col else np.zeros(0, np.int32),
            np.concatenate(out_val) if out_val else np.zeros(0), total_nnz, total_products, len(bounds) - 1)


def check_config(g, name, n_random, n_heaviest):
    A = wl.CONFIGS[name].make()
    ip = oracle.row_products(A, A)
    rows = sample_rows(ip, n_random, n_heaviest, seed=len(name))
    rp, col, val, nnz, products, panels = run_sampled(g, A, rows)
    assert products == int(ip.sum())
    ref = oracle.spgemm(A, A, rows=rows)
    worst = compare_rows(np.arange(rows.size), rp, col, val, ref)
    print("%s: panels=%d products=%d nnz(C)=%d sampled_rows=%d max_rel_err=%.2e" % (
        name, panels, products, nnz, rows.size, worst))
    return A, ip, nnz


def test_banded20_full(g):
    A, ip, nnz = check_config(g, "banded20", 3000, 5)
    n = A.n_rows
    assert A.nnz == 27 * n - 182 and int(ip.sum()) == 729 * n - 8190 and nnz == 53 * n - 702


def test_er22_full(g):
    A, ip, nnz = check_config(g, "er22", 3000, 5)
    assert int(ip.sum()) == 1 << 30 and np.all(ip == 256)
    # distinct columns per row can only shrink from 256 through collisions
    assert (1 << 30) - 100_000 < nnz <= 1 << 30


def test_rmat22_full(g):
    check_config(g, "rmat22", 400, 3)


def test_rmat23_full(g):
    check_config(g, "rmat23", 400, 3)


def test_rmat20_pair_full(g):
    # C = A*B, R-MAT scale 20 with A edge factor 32 and B edge factor 8
    A, B = wl.PAIRS["rmat20_a32_b8"].make()
    ip = oracle.row_products(A, B)
    rows = sample_rows(ip, 400, 3, seed=20)
    rp, col, val, nnz, products, panels = run_sampled(g, A, rows, B=B)
    assert products == int(ip.sum())
    ref = oracle.spgemm(A, B, rows=rows)
    worst = compare_rows(np.arange(rows.size), rp, col, val, ref)
    print("rmat20_a32_b8: panels=%d products=%d nnz(C)=%d sampled_rows=%d max_rel_err=%.2e" % (
        panels, products, nnz, rows.size, worst))


def test_rmat20_pair_pattern_reuse_full(g):
    # the same pair at full size, every panel recomputed for new values of A
    # and B on its kept pattern; sampled rows against the oracle's for the new values
    A, B = wl.PAIRS["rmat20_a32_b8"].make()
    rng = np.random.default_rng(21)
    A2 = A.with_values(rng.uniform(-1.0, 1.0, A.nnz))
    B2 = B.with_values(rng.uniform(-1.0, 1.0, B.nnz))
    ip = oracle.row_products(A, B)
    rows = sample_rows(ip, 300, 3, seed=21)
    rp, col, val, nnz, products, panels = run_sampled(g, A, rows, B=B, new_values=(A2.val, B2.val))
    assert products == int(ip.sum())
    worst = compare_rows(np.arange(rows.size), rp, col, val, oracle.spgemm(A2, B2, rows=rows))
    print("rmat20_a32_b8 new values: panels=%d nnz(C)=%d sampled_rows=%d max_rel_err=%.2e" % (
        panels, nnz, rows.size, worst))
