"""Parity of the HIP SpGEMM (through the C ABI) with the CPU oracle, on
seeded inputs small enough for the oracle to finish in seconds while still
spanning many tiles and ragged tails, and on the corner cases of the method
(empty rows/columns, forced multisplit depths, panels, explicit zeros)."""
import numpy as np
import pytest

import oracle
import workloads as wl
from tests.parity import compare_full, compare_rows

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def g():
    from paper_2607_22866_amd import gmagnus

    gmagnus.load()
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return gmagnus


def run(g, A, B, **opts):
    dA = g.DeviceCSR.from_host(A)
    dB = dA if B is A else g.DeviceCSR.from_host(B)
    with g.Plan(dA, dB, **opts) as p:
        rp, nnz = p.symbolic()
        col, val = p.numeric()
        info = p.info()
    torch.cuda.synchronize()
    assert info.check_flags == 0, info.check_flags
    return rp.cpu().numpy(), col.cpu().numpy(), val.cpu().numpy(), info


def check(g, A, B, **opts):
    rp, col, val, info = run(g, A, B, **opts)
    r0 = opts.get("row_begin", 0)
    r1 = opts.get("row_end", 0) or A.n_rows
    ref = oracle.spgemm(A, B, rows=np.arange(r0, r1))
    compare_full(rp, col, val, ref)
    return info


RMAT12 = wl.CONFIGS["rmat12"]

# (tau, dense_width_log2, chunks_max_log2) -> expected multisplit levels for C.m = 4096
DEPTHS = [
    ({}, []),
    (dict(tau=600, dense_width_log2=8, chunks_max_log2=4), [16]),
    (dict(tau=300, dense_width_log2=7, chunks_max_log2=3), [8, 4]),
    (dict(tau=200, dense_width_log2=6, chunks_max_log2=2), [4, 4, 4]),
    (dict(tau=150, dense_width_log2=5, chunks_max_log2=5), [32, 4]),
    (dict(tau=128, dense_width_log2=5, chunks_max_log2=1), [2, 2, 2, 2, 2, 2, 2]),
]


@pytest.mark.parametrize("opts,levels", DEPTHS)
def test_rmat12_every_depth(g, opts, levels):
    A = RMAT12.make()
    info = check(g, A, A, **opts)
    assert info.params.levels == levels
    ip = oracle.row_products(A, A)
    # rows are heavy above min(tau, 3456) products (the light accumulators'
    # efficient range); chunks are classified by tau
    tau = info.params.tau
    assert info.row_tau == min(tau, 3456)
    assert info.n_heavy_rows == int((ip > info.row_tau).sum())
    assert info.products_total == int(ip.sum())
    assert info.products_heavy == int(ip[ip > info.row_tau].sum())
    # nnz(C) and the heavy rows' share of it, from the oracle's row counts
    cnt = oracle.row_counts(A, A)
    assert info.c_nnz == int(cnt.sum())
    assert info.c_nnz_heavy == int(cnt[ip > info.row_tau].sum())
    if levels:
        assert info.levels_run >= 1


@pytest.mark.parametrize("opts,levels", DEPTHS[1:])
def test_rmat12_paper_histogram(g, opts, levels):
    # the level-0 histogram as a pass over C-hat's columns gives the same C
    A = RMAT12.make()
    info = check(g, A, A, flags=g.FLAG_PAPER_HISTOGRAM, **opts)
    assert info.params.levels == levels


@pytest.mark.parametrize("opts,levels", DEPTHS[1:])
def test_rmat12_paper_expansion(g, opts, levels):
    # C-hat written row by row and split at level 0 by the multisplit (the
    # paper's order) gives the same C as the split fused into the expansion
    A = RMAT12.make()
    info = check(g, A, A, flags=g.FLAG_PAPER_EXPANSION, **opts)
    assert info.params.levels == levels


@pytest.mark.parametrize("opts,levels", DEPTHS[1:])
def test_rmat12_slice_order_split(g, opts, levels):
    # the first-level split done during a slice-order expansion (runs at
    # atomic cursors) gives the same C as the chunk-major row-order one
    A = RMAT12.make()
    info = check(g, A, A, flags=g.FLAG_SLICE_SPLIT, **opts)
    assert info.params.levels == levels


@pytest.mark.parametrize("opts,levels", [d for d in DEPTHS if len(d[1]) == 2])
def test_rmat12_two_levels_level_by_level(g, opts, levels):
    # with two levels the expansion writes the final chunks directly; writing
    # the first level out and splitting it in its own pass gives the same C
    A = RMAT12.make()
    info = check(g, A, A, flags=g.FLAG_LEVEL_BY_LEVEL, **opts)
    assert info.params.levels == levels and info.levels_run == 2


def test_rmat12_integer_values_bit_exact(g):
    A = wl.rmat(12, 8, 0.57, 0.19, 0.19, 12, values="int3")
    for opts in ({}, dict(tau=200, dense_width_log2=6, chunks_max_log2=2),
                 dict(tau=200, dense_width_log2=6, chunks_max_log2=2, flags=g.FLAG_PAPER_EXPANSION),
                 dict(tau=200, dense_width_log2=6, chunks_max_log2=2, flags=g.FLAG_SLICE_SPLIT),
                 dict(tau=300, dense_width_log2=7, chunks_max_log2=3),
                 dict(tau=300, dense_width_log2=7, chunks_max_log2=3, flags=g.FLAG_LEVEL_BY_LEVEL)):
        rp, col, val, _ = run(g, A, A, **opts)
        ref = oracle.spgemm(A, A)
        assert np.array_equal(rp, ref.row_ptr) and np.array_equal(col, ref.col)
        assert np.array_equal(val, ref.val)  # exact integers in any summation order


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_rmat_scales(g, seed):
    A = wl.rmat(13 + seed % 2, 8 + 4 * seed, 0.57, 0.19, 0.19, 40 + seed)
    check(g, A, A)
    check(g, A, A, tau=256, dense_width_log2=7, chunks_max_log2=3)


@pytest.mark.parametrize("chunks_max_log2,levels", [(2, [4, 2]), (1, [2, 2, 2])])
def test_wide_final_chunks(g, chunks_max_log2, levels):
    # 2^16 columns with at most 4 (or 2) chunks per level: the first level's
    # light chunks are final and wider than the dense width, so the wide
    # accumulators run (bitmap rank, the small-chunk sort, hashing); with two
    # levels the fused expansion writes them, with three the row-order one
    A = wl.rmat(16, 4, 0.57, 0.19, 0.19, 16)
    info = check(g, A, A, tau=300, chunks_max_log2=chunks_max_log2)
    assert info.params.levels == levels


def test_first_level_chunks_of_2_18_columns(g):
    # 2^19 columns, at most 2 chunks per level: the first level's light chunks
    # span 2^18 columns, which the bitmap-rank kernels cover in two halves
    A = wl.rmat(19, 2, 0.57, 0.19, 0.19, 19)
    info = check(g, A, A, tau=300, chunks_max_log2=1, row_begin=0, row_end=65536)
    assert info.params.levels[0] == 2 and info.levels_run >= 2


def test_distinct_a_b_non_square(g):
    A = wl.rmat(11, 8, 0.57, 0.19, 0.19, 7)
    B = wl.erdos_renyi(A.n_cols, 3000, 12, 8)  # 2048 x 3000, C.m not a power of two
    check(g, A, B)
    check(g, A, B, tau=300, dense_width_log2=6, chunks_max_log2=3)


@pytest.mark.parametrize("a_ef,b_ef", [(4, 4), (4, 16), (16, 8), (64, 16)])
def test_rmat_pair_grid(g, a_ef, b_ef):
    # C = A*B with two R-MAT matrices of scale 15 and different densities
    # (the paper's RMat grid, Section IV-A, at a size the oracle finishes);
    # every row is compared, with the planner's depth and with a forced
    # two-level split
    A = wl.rmat(15, a_ef, 0.57, 0.19, 0.19, 1000 + a_ef)
    B = wl.rmat(15, b_ef, 0.57, 0.19, 0.19, 1001 + b_ef)
    check(g, A, B)
    if a_ef == 16:
        info = check(g, A, B, tau=2048, dense_width_log2=9, chunks_max_log2=3)
        assert len(info.params.levels) >= 2


@pytest.mark.parametrize("shape,density", [((1, 1, 1), 1.0), ((37, 50, 61), 0.1), ((200, 300, 150), 0.05),
                                           ((64, 64, 64), 0.0), ((130, 5, 700), 0.5)])
def test_uniform_small(g, shape, density):
    m, k, n = shape
    A = wl.uniform(m, k, density, m + k)
    B = wl.uniform(k, n, density, n + 7)
    check(g, A, B)
    check(g, A, B, tau=128, dense_width_log2=5, chunks_max_log2=2)


def test_banded_window_and_hash(g):
    A = wl.banded(4096, 13, 3)
    info = check(g, A, A)
    assert info.n_heavy_rows == 0
    check(g, A, A, flags=4)  # hash accumulator instead of the dense window
    W = wl.banded(3000, 300, 4)  # 601-wide rows: wider window bin
    check(g, W, W)


def _drop_rows(A, rows):
    """A with the given rows emptied (host CSR surgery for edge cases)."""
    keep = np.ones(A.n_rows, dtype=bool)
    keep[rows] = False
    lens = np.diff(A.row_ptr) * keep
    rp = np.zeros(A.n_rows + 1, dtype=np.int64)
    rp[1:] = np.cumsum(lens)
    mask = np.repeat(keep, np.diff(A.row_ptr))
    return wl.CSR(A.n_rows, A.n_cols, rp, np.ascontiguousarray(A.col[mask]), np.ascontiguousarray(A.val[mask]))


def _stack_rows(X, Y):
    """Rows of X followed by rows of Y (same column count)."""
    rp = np.concatenate([X.row_ptr, X.row_ptr[-1] + Y.row_ptr[1:]])
    return wl.CSR(X.n_rows + Y.n_rows, X.n_cols, rp, np.concatenate([X.col, Y.col]), np.concatenate([X.val, Y.val]))


def test_narrow_windows(g):
    # rows spanning at most 64 columns: with many of them the symbolic counts
    # come from per-B-row column masks, with few from the per-product window;
    # empty B rows reached from narrow rows add nothing
    A = _drop_rows(wl.banded(3000, 9, 7), np.arange(100, 400, 3))
    info = check(g, A, A)
    assert info.n_heavy_rows == 0
    B = _drop_rows(wl.banded(3000, 20, 8), np.arange(0, 3000, 5))
    check(g, A, B)
    # a few narrow rows among wide ones (fewer than an eighth of B's rows:
    # the per-product window kernel)
    Nb = wl.banded(3000, 9, 9)
    top = wl.CSR(300, 3000, Nb.row_ptr[:301].copy(), Nb.col[:Nb.row_ptr[300]].copy(), Nb.val[:Nb.row_ptr[300]].copy())
    M = _stack_rows(top, wl.erdos_renyi(3 * 3000, 3000, 12, 10))
    N = wl.banded(3000, 9, 11)
    check(g, M, N)


def test_erdos_renyi(g):
    A = wl.erdos_renyi(1 << 14, 1 << 14, 16, 5)
    info = check(g, A, A)
    assert info.products_total == 256 << 14


def test_identity_permutation_exact(g):
    A = RMAT12.make()
    I = wl.identity(A.n_rows)
    for X, Y in ((I, A), (A, I)):
        rp, col, val, _ = run(g, X, Y)
        assert np.array_equal(rp, A.row_ptr) and np.array_equal(col, A.col) and np.array_equal(val, A.val)
    P = wl.permutation(A.n_rows, 9)
    rp, col, val, _ = run(g, P, A)
    perm = P.col.astype(np.int64)
    for i in range(0, A.n_rows, 11):
        s, e = A.row_ptr[perm[i]], A.row_ptr[perm[i] + 1]
        assert np.array_equal(col[rp[i]:rp[i + 1]], A.col[s:e])
        assert np.array_equal(val[rp[i]:rp[i + 1]], A.val[s:e])


def test_structural_zeros_kept(g):
    A = wl.CSR(2, 2, np.array([0, 2, 3], np.int64), np.array([0, 1, 1], np.int32), np.array([1.0, -1.0, 2.0]))
    B = wl.CSR(2, 3, np.array([0, 2, 3], np.int64), np.array([0, 2, 2], np.int32), np.array([5.0, 2.0, 2.0]))
    rp, col, val, _ = run(g, A, B)
    assert list(rp) == [0, 2, 3] and list(col) == [0, 2, 2] and list(val) == [5.0, 0.0, 4.0]
    # the same cancellation inside a heavy row (forced with a small tau)
    H = wl.rmat(10, 16, 0.57, 0.19, 0.19, 2, values="int3")
    check(g, H, H, tau=128, dense_width_log2=6, chunks_max_log2=2)


def test_empty_and_degenerate(g):
    E = wl.empty(50, 40)
    B = wl.uniform(40, 30, 0.2, 1)
    rp, col, val, info = run(g, E, B)
    assert np.all(rp == 0) and col.size == 0
    A = wl.uniform(30, 40, 0.2, 2)
    rp, col, val, info = run(g, A, wl.empty(40, 30))
    assert np.all(rp == 0) and info.products_total == 0
    one = wl.uniform(1, 1, 1.0, 3)
    check(g, one, one)
    # a row panel with no rows
    R = RMAT12.make()
    rp, col, val, _ = run(g, R, R, row_begin=100, row_end=100)
    assert list(rp) == [0] and col.size == 0


def test_panels_concatenate_to_full(g):
    A = RMAT12.make()
    dA = g.DeviceCSR.from_host(A)
    bounds = g.split_panels(dA, dA, 200_000)
    assert bounds[0] == 0 and bounds[-1] == A.n_rows and len(bounds) > 3
    ip = oracle.row_products(A, A)
    pre = np.concatenate([[0], np.cumsum(ip)])
    for a, b in zip(bounds[:-1], bounds[1:]):
        assert pre[b] - pre[a] <= 200_000 or b == a + 1
    ref = oracle.spgemm(A, A)
    for a, b in zip(bounds[:-1], bounds[1:]):
        rp, col, val, _ = run(g, A, A, row_begin=a, row_end=b)
        assert np.array_equal(rp + ref.row_ptr[a], ref.row_ptr[a:b + 1])
        s, e = ref.row_ptr[a], ref.row_ptr[b]
        assert np.array_equal(col, ref.col[s:e])
        assert np.all(np.abs(val - ref.val[s:e]) <= 1e-12 * ref.bound[s:e])


def greedy_panels(pre, max_products):
    """The split the header specifies: from row r, the furthest end e with
    pre[e] - pre[r] <= max_products, at least one row."""
    n = pre.size - 1
    out, r = [0], 0
    while r < n:
        e = int(np.searchsorted(pre, pre[r] + max_products, side="right")) - 1
        r = max(e, r + 1)
        out.append(r)
    return out


def test_split_panels_greedy_bounds(g):
    # exact bounds for limits from one row per panel (4096 panels: more than
    # one read of the bounds) to a single panel, with empty rows in between
    A = wl.rmat(12, 8, 0.57, 0.19, 0.19, 12)
    dA = g.DeviceCSR.from_host(A)
    pre = np.concatenate([[0], np.cumsum(oracle.row_products(A, A))])
    # the limits around nnz(A) * (longest B row) take the one-panel shortcut
    # on one side and the row products on the other
    bound = int(A.nnz) * int(np.diff(A.row_ptr).max())
    for mp in (1, 37, 5_000, 200_000, int(pre[-1]) - 1, int(pre[-1]), bound - 1, bound, 1 << 40):
        assert g.split_panels(dA, dA, mp) == greedy_panels(pre, mp), mp
    n_need = len(greedy_panels(pre, 5_000)) - 1
    assert len(g.split_panels(dA, dA, 5_000, max_panels=n_need)) == n_need + 1
    with pytest.raises(g.GmagnusError):
        g.split_panels(dA, dA, 5_000, max_panels=n_need - 1)


def test_row_products_abi(g):
    A = wl.rmat(13, 16, 0.57, 0.19, 0.19, 77)
    dA = g.DeviceCSR.from_host(A)
    ip = g.row_products(dA, dA).cpu().numpy()
    assert np.array_equal(ip, oracle.row_products(A, A))


def test_validate_flags_bad_csr(g):
    A = wl.uniform(20, 20, 0.3, 5)
    bad = wl.CSR(A.n_rows, A.n_cols, A.row_ptr.copy(), A.col.copy(), A.val.copy())
    r = int(np.argmax(np.diff(bad.row_ptr) >= 2))
    s = bad.row_ptr[r]
    bad.col[s], bad.col[s + 1] = bad.col[s + 1], bad.col[s]  # unsorted row
    dA = g.DeviceCSR.from_host(bad)
    with pytest.raises(g.GmagnusError) as e:
        g.Plan(dA, dA, validate=1)
    assert e.value.status == 2
    g.Plan(g.DeviceCSR.from_host(A), g.DeviceCSR.from_host(A), validate=1).close()


def test_numeric_before_symbolic_rejected(g):
    A = RMAT12.make()
    dA = g.DeviceCSR.from_host(A)
    with g.Plan(dA, dA) as p:
        p.nnz = 0
        p.row_ptr = torch.zeros(A.n_rows + 1, dtype=torch.int64, device="cuda")
        with pytest.raises(g.GmagnusError) as e:
            p.numeric(torch.empty(1, dtype=torch.int32, device="cuda"), torch.empty(1, dtype=torch.float64,
                                                                                    device="cuda"))
        assert e.value.status == 4


@pytest.mark.parametrize("opts", [dict(), dict(tau=300, dense_width_log2=7, chunks_max_log2=3)])
def test_concurrent_streams(g, opts):
    # heavy and light rows on two streams joined by events give the same C
    A = RMAT12.make()
    check(g, A, A, flags=g.FLAG_CONCURRENT_STREAMS, **opts)


def test_serial_streams_and_timing_flags(g):
    A = RMAT12.make()
    # three levels: the levels after the first run the multisplit kernel
    info = check(g, A, A, flags=1 | 2, tau=200, dense_width_log2=6, chunks_max_log2=2)
    d = info.to_dict()
    assert d["kernels"]["expand"]["ms"] > 0 and d["kernels"]["multisplit"]["launches"] >= 1
    # two levels: both are written by the expansion, no multisplit pass
    info = check(g, A, A, flags=1 | 2, tau=300, dense_width_log2=7, chunks_max_log2=3)
    d = info.to_dict()
    assert d["kernels"]["multisplit"]["launches"] == 0 and info.levels_run == 2
    info = check(g, A, A, flags=1 | 2 | g.FLAG_LEVEL_BY_LEVEL, tau=300, dense_width_log2=7, chunks_max_log2=3)
    assert info.to_dict()["kernels"]["multisplit"]["launches"] == 1


def test_sampled_rows_helper(g):
    A = wl.rmat(14, 8, 0.57, 0.19, 0.19, 5)
    rp, col, val, _ = run(g, A, A)
    rows = np.random.default_rng(0).choice(A.n_rows, 300, replace=False)
    compare_rows(rows, rp, col, val, oracle.spgemm(A, A, rows=rows))


REUSE_CASES = [
    ("no split", 0, {}),
    ("one level", 0, dict(tau=600, dense_width_log2=8, chunks_max_log2=4)),
    ("two levels in one pass", 0, dict(tau=300, dense_width_log2=7, chunks_max_log2=3)),
    ("three levels", 0, dict(tau=200, dense_width_log2=6, chunks_max_log2=2)),
    ("paper order", 16, dict(tau=200, dense_width_log2=6, chunks_max_log2=2)),
    ("slice order", 32, dict(tau=300, dense_width_log2=7, chunks_max_log2=3)),
    ("level by level", 64, dict(tau=300, dense_width_log2=7, chunks_max_log2=3)),
    # the replay runs on the heavy rows' own stream, joined to the plan's by events
    ("two streams", 128, dict(tau=300, dense_width_log2=7, chunks_max_log2=3)),
]


@pytest.mark.parametrize("name,flags,opts", REUSE_CASES, ids=[c[0] for c in REUSE_CASES])
@pytest.mark.parametrize("same", [True, False], ids=["A*A", "A*B"])
def test_pattern_reuse(g, name, flags, opts, same):
    # symbolic once, then numeric for three value sets on the same patterns
    # (new values through gmagnus_update_values): each C equals the oracle's
    # for that value set, on the structure the first symbolic produced
    A = RMAT12.make()
    B = A if same else wl.rmat(12, 4, 0.57, 0.19, 0.19, 77)
    dA = g.DeviceCSR.from_host(A)
    dB = dA if same else g.DeviceCSR.from_host(B)
    rng = np.random.default_rng(5)
    with g.Plan(dA, dB, flags=flags | g.FLAG_KEEP_PATTERN, **opts) as p:
        rp, nnz = p.symbolic()
        rp_h = rp.cpu().numpy()
        for it in range(3):
            if it == 0:
                A2, B2 = A, B
            else:
                A2 = A.with_values(rng.uniform(-1.0, 1.0, A.nnz))
                B2 = A2 if same else B.with_values(rng.uniform(-1.0, 1.0, B.nnz))
                va = torch.from_numpy(A2.val).cuda()
                vb = va if same else torch.from_numpy(B2.val).cuda()
                p.update_values(va, None if same else vb)
            col, val = p.numeric()
            info = p.info()
            torch.cuda.synchronize()
            assert info.check_flags == 0, info.check_flags
            compare_full(rp_h, col.cpu().numpy(), val.cpu().numpy(), oracle.spgemm(A2, B2))
        if opts:
            assert info.levels_run >= 1


def test_update_values_errors(g):
    A = RMAT12.make()
    dA = g.DeviceCSR.from_host(A)
    with g.Plan(dA, dA, tau=300, dense_width_log2=7, chunks_max_log2=3) as p:
        p.symbolic()
        with pytest.raises(g.GmagnusError):
            p.update_values(dA.val)  # plan made without FLAG_KEEP_PATTERN
    with g.Plan(dA, dA, flags=g.FLAG_KEEP_PATTERN) as p:
        with pytest.raises(g.GmagnusError):
            p.update_values(dA.val)  # before symbolic


class _CountingAllocator:
    """Device workspace through torch's caching allocator; call number
    `fail_at` (1-based) returns NULL. Tracks the blocks still outstanding."""

    def __init__(self, g, fail_at=0):
        self.fail_at, self.calls, self.live = fail_at, 0, set()
        self.alloc = g.ALLOC_FN(self._alloc)
        self.free = g.FREE_FN(self._free)

    def _alloc(self, nbytes, stream, ctx):
        self.calls += 1
        if self.calls == self.fail_at:
            return None
        p = torch.cuda.caching_allocator_alloc(nbytes)
        self.live.add(p)
        return p

    def _free(self, ptr, stream, ctx):
        self.live.discard(ptr)
        torch.cuda.caching_allocator_delete(ptr)


def _run_with_allocator(g, dA, al, **opts):
    """plan + symbolic + numeric with the allocator; returns (status, C or None)."""
    try:
        with g.Plan(dA, dA, alloc=al.alloc, free=al.free, **opts) as p:
            rp, nnz = p.symbolic()
            col, val = p.numeric()
            info = p.info()
            torch.cuda.synchronize()
            assert info.check_flags == 0
            return 0, (rp.cpu().numpy(), col.cpu().numpy(), val.cpu().numpy())
    except g.GmagnusError as e:
        return e.status, None


@pytest.mark.parametrize("opts", [dict(), dict(tau=300, dense_width_log2=7, chunks_max_log2=3)],
                         ids=["default", "two levels"])
def test_user_allocator_failure_releases_everything(g, opts):
    # a user allocator that returns NULL on its N-th call: the call that needed
    # the block fails with OUT_OF_MEMORY, and every block handed out before is
    # given back once the plan is destroyed (nothing leaks); without a failure
    # the same allocator gives the oracle's C
    A = RMAT12.make()
    dA = g.DeviceCSR.from_host(A)
    ok = _CountingAllocator(g)
    st, C = _run_with_allocator(g, dA, ok, **opts)
    assert st == 0 and not ok.live
    compare_full(*C, oracle.spgemm(A, A))
    total = ok.calls
    assert total >= 10
    for n in sorted({1, 2, 3, total // 4, total // 2, total - 1, total}):
        al = _CountingAllocator(g, fail_at=n)
        st, _ = _run_with_allocator(g, dA, al, **opts)
        assert st == 3, (n, st)
        assert not al.live, "call %d failed: %d blocks not given back" % (n, len(al.live))
    torch.cuda.synchronize()


def test_workspace_limit(g):
    A = RMAT12.make()
    dA = g.DeviceCSR.from_host(A)
    opts = dict(tau=300, dense_width_log2=7, chunks_max_log2=3)
    with g.Plan(dA, dA, **opts) as p:
        p.symbolic()
        p.numeric()
        peak = p.info().workspace_peak_bytes
    assert peak > 0
    # a limit below what the plan needs fails cleanly
    with pytest.raises(g.GmagnusError) as e:
        with g.Plan(dA, dA, workspace_limit_bytes=peak // 4, **opts) as p:
            p.symbolic()
            p.numeric()
    assert e.value.status == 3 and "workspace limit" in str(e.value)
    # at the peak it runs, stays within the limit and gives the oracle's C
    info = check(g, A, A, workspace_limit_bytes=peak, **opts)
    assert 0 < info.workspace_peak_bytes <= peak


def test_timed_classes_fit_in_wall_time(g):
    # the per-class device times of one plan do not overlap: their sum stays
    # within the wall time of the calls that produced them
    import time

    A = wl.rmat(15, 16, 0.57, 0.19, 0.19, 3)
    dA = g.DeviceCSR.from_host(A)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    with g.Plan(dA, dA, flags=g.FLAG_TIMING) as p:
        p.symbolic()
        p.numeric()
        torch.cuda.synchronize()
        wall_ms = 1000.0 * (time.perf_counter() - t0)
        info = p.info()
    total = sum(info.kernel_ms[i] for i in range(len(g.K_NAMES)))
    assert info.expansion_path == 3  # one level (C.m = 2^15), split during the row-order expansion
    assert 0 < total <= wall_ms, (total, wall_ms)
    assert info.kernel_ms[2] > 0 and info.kernel_ms[6] > 0


@pytest.mark.parametrize("kind", ["read", "read_nt", "write", "write_nt", "copy", "gather"])
def test_bandwidth_probe(g, kind):
    import ctypes

    n = 1 << 22
    src = torch.arange(n, dtype=torch.float64, device="cuda")
    dst = torch.full((n,), -7.0, dtype=torch.float64, device="cuda")
    ms = ctypes.c_double()
    st = g.load().gmagnus_bandwidth_probe(g.PROBE_KINDS[kind], dst.data_ptr(), src.data_ptr(), 8 * n, 0, 3,
                                          torch.cuda.current_stream().cuda_stream, ctypes.byref(ms))
    assert st == 0 and ms.value > 0
    if kind == "copy":
        assert torch.equal(dst, src)
    elif kind.startswith("write"):
        # element i of 16 bytes holds (1.0, i)
        assert torch.equal(dst[0::2], torch.ones(n // 2, dtype=torch.float64, device="cuda"))
        assert torch.equal(dst[1::2], torch.arange(n // 2, dtype=torch.float64, device="cuda"))
    else:
        assert torch.equal(dst, torch.full((n,), -7.0, dtype=torch.float64, device="cuda"))  # sink untouched
    assert 10.0 < g.bandwidth_probe(kind, nbytes=1 << 28) < 20000.0
    if kind == "gather":  # the working set must be a power of two
        st = g.load().gmagnus_bandwidth_probe(g.PROBE_KINDS[kind], dst.data_ptr(), src.data_ptr(), 3 << 20, 0, 1,
                                              torch.cuda.current_stream().cuda_stream, ctypes.byref(ms))
        assert st == 1
