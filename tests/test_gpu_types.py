"""Type variants of the HIP SpGEMM (fp32 values, int64 column indices; the
s_col / s_val of the paper's parameter selection, Section III-D) against the
oracle: structure exact, values within the fp64 bar or, for fp32, within
(n + 1) * 2^-24 * sum |ab| per entry (tests/parity.py)."""
import numpy as np
import pytest

import oracle
import workloads as wl
from tests.parity import compare_full

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TYPES = [(torch.int32, torch.float32), (torch.int64, torch.float64), (torch.int64, torch.float32)]
TYPE_IDS = ["i32-f32", "i64-f64", "i64-f32"]

DEPTHS = [
    ({}, None),
    (dict(tau=600, dense_width_log2=8, chunks_max_log2=4), [16]),
    (dict(tau=300, dense_width_log2=7, chunks_max_log2=3), [8, 4]),
    (dict(tau=200, dense_width_log2=6, chunks_max_log2=2), [4, 4, 4]),
    (dict(tau=150, dense_width_log2=5, chunks_max_log2=5), [32, 4]),
]


@pytest.fixture(scope="module")
def g():
    from paper_2607_22866_amd import gmagnus

    gmagnus.load()
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return gmagnus


def as_type(M, vdt):
    """The matrix the GPU sees: values rounded to fp32 when vdt is float32."""
    if vdt == torch.float32:
        return M.with_values(M.val.astype(np.float32).astype(np.float64))
    return M


def run_typed(g, A, B, idt, vdt, **opts):
    dA = g.DeviceCSR.from_host(A, index_dtype=idt, value_dtype=vdt)
    dB = dA if B is A else g.DeviceCSR.from_host(B, index_dtype=idt, value_dtype=vdt)
    with g.Plan(dA, dB, **opts) as p:
        rp, nnz = p.symbolic()
        col, val = p.numeric()
        info = p.info()
    torch.cuda.synchronize()
    assert info.check_flags == 0, info.check_flags
    assert col.dtype == idt and val.dtype == vdt
    assert info.index_type == g.INDEX_TYPES[idt] and info.value_type == g.VALUE_TYPES[vdt]
    return rp.cpu().numpy(), col.cpu().numpy(), val.cpu().numpy(), info


def check_typed(g, A, B, idt, vdt, **opts):
    A2 = as_type(A, vdt)
    B2 = A2 if B is A else as_type(B, vdt)
    rp, col, val, info = run_typed(g, A2, B2, idt, vdt, **opts)
    compare_full(rp, col, val, oracle.spgemm(A2, B2), f32=vdt == torch.float32)
    return info


@pytest.mark.parametrize("types", TYPES, ids=TYPE_IDS)
@pytest.mark.parametrize("opts,levels", DEPTHS, ids=["derived", "1", "2", "3", "32x4"])
def test_rmat12_types_every_depth(g, types, opts, levels):
    idt, vdt = types
    A = wl.CONFIGS["rmat12"].make()
    info = check_typed(g, A, A, idt, vdt, **opts)
    p = g.get_params(A.n_cols, 163840, idt, vdt, **opts)
    assert info.params.tau == p.tau and info.params.levels == p.levels
    if levels is not None:
        assert info.params.levels == levels and info.levels_run == len(levels)


@pytest.mark.parametrize("types", TYPES, ids=TYPE_IDS)
def test_light_rows_types(g, types):
    # dense window (banded), hash and sort bins (ER, uniform)
    idt, vdt = types
    for A in (wl.banded(20000, 13, 3), wl.erdos_renyi(20000, 20000, 16, 4), wl.uniform(3000, 3000, 0.01, 5)):
        check_typed(g, A, A, idt, vdt)


@pytest.mark.parametrize("types", TYPES, ids=TYPE_IDS)
def test_rmat_pair_types(g, types):
    idt, vdt = types
    A = wl.rmat(13, 8, 0.57, 0.19, 0.19, 6)
    B = wl.rmat(13, 4, 0.57, 0.19, 0.19, 7)
    check_typed(g, A, B, idt, vdt)


@pytest.mark.parametrize("vdt", [torch.float64, torch.float32], ids=["f64", "f32"])
def test_int64_columns_beyond_2_31(g, vdt):
    # C with 3 * 2^30 columns: rows whose columns spread over the whole range
    # go to the heavy path (chunk-local columns fit 32 bits), rows whose
    # columns stay inside a window remain light rows keyed by offsets from
    # their smallest column
    n_cols = 3 << 30
    A = wl.uniform(300, 400, 0.03, 8)
    cases = ((wl.wide(400, n_cols, 12, 9), True),
             (wl.wide(400, n_cols, 12, 10, window=50000, base=(1 << 31) + 12345), False),
             (wl.wide(400, n_cols, 12, 15, window=1000, base=(3 << 30) - 1000), False))
    for B, heavy in cases:
        info = check_typed(g, A, B, torch.int64, vdt)
        assert (info.n_heavy_rows > 0) == heavy
        assert info.params.levels == g.get_params(n_cols, 163840, torch.int64, vdt).levels
        assert info.c_nnz > 0


def test_int64_columns_paper_order_refused(g):
    n_cols = 3 << 30
    A = wl.uniform(100, 50, 0.05, 11)
    B = wl.wide(50, n_cols, 10, 12)
    dA = g.DeviceCSR.from_host(A, index_dtype=torch.int64)
    dB = g.DeviceCSR.from_host(B, index_dtype=torch.int64)
    with pytest.raises(g.GmagnusError) as e:
        with g.Plan(dA, dB, flags=g.FLAG_PAPER_EXPANSION) as p:
            p.symbolic()
    assert e.value.status == 6


@pytest.mark.parametrize("opts", [{}, dict(tau=300, dense_width_log2=7, chunks_max_log2=3)], ids=["derived", "2"])
def test_pattern_reuse_fp32(g, opts):
    A = as_type(wl.CONFIGS["rmat12"].make(), torch.float32)
    dA = g.DeviceCSR.from_host(A, value_dtype=torch.float32)
    rng = np.random.default_rng(13)
    with g.Plan(dA, dA, flags=g.FLAG_KEEP_PATTERN, **opts) as p:
        rp, _ = p.symbolic()
        rp_h = rp.cpu().numpy()
        for it in range(2):
            A2 = as_type(A.with_values(rng.uniform(-1.0, 1.0, A.nnz)), torch.float32)
            p.update_values(torch.from_numpy(A2.val.astype(np.float32)).cuda())
            col, val = p.numeric()
            torch.cuda.synchronize()
            assert p.info().check_flags == 0
            compare_full(rp_h, col.cpu().numpy(), val.cpu().numpy(), oracle.spgemm(A2, A2), f32=True)


def test_typed_errors(g):
    import ctypes

    A = wl.rmat(10, 4, 0.57, 0.19, 0.19, 14)
    d32 = g.DeviceCSR.from_host(A)
    d64 = g.DeviceCSR.from_host(A, index_dtype=torch.int64)
    df32 = g.DeviceCSR.from_host(A, value_dtype=torch.float32)
    with pytest.raises(g.GmagnusError) as e:
        g.Plan(d32, d64)
    assert e.value.status == 1
    with pytest.raises(g.GmagnusError) as e:
        g.Plan(d32, df32)
    assert e.value.status == 1
    # the untyped numeric and update_values refuse plans of other types
    with g.Plan(df32, df32) as p:
        rp, nnz = p.symbolic()
        col = torch.empty(nnz, dtype=torch.int32, device="cuda")
        val = torch.empty(nnz, dtype=torch.float64, device="cuda")
        st = g.load().gmagnus_spgemm_numeric(p._h, rp.data_ptr(), col.data_ptr(), val.data_ptr())
        assert st == 1
        with pytest.raises(ValueError):
            p.update_values(torch.zeros(A.nnz, dtype=torch.float64, device="cuda"))
    del ctypes
