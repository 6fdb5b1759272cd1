"""gmagnus_plan_static: the plan whose device workspace is the library's static
device array (for callers that cannot allocate). Its C must equal
gmagnus_plan's: row pointers and columns bit for bit, values within the
oracle's tolerance, on two calls in a row with the second input smaller (the
array keeps the first call's contents), and the oracle's C itself."""
import numpy as np
import pytest

import oracle
import workloads as wl
from tests.parity import TOL, compare_full

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def g():
    from paper_2607_22866_amd import gmagnus

    gmagnus.load()
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return gmagnus


def _product(g, dA, dB, static, **opts):
    with g.Plan(dA, dB, static_workspace=static, **opts) as p:
        rp, nnz = p.symbolic()
        col, val = p.numeric()
        info = p.info()
    torch.cuda.synchronize()
    assert info.check_flags == 0
    return rp.cpu().numpy(), col.cpu().numpy(), val.cpu().numpy(), info


OPTS = [dict(), dict(tau=300, dense_width_log2=7, chunks_max_log2=3), dict(tau=200, dense_width_log2=6,
                                                                           chunks_max_log2=2)]


@pytest.mark.parametrize("opts", OPTS, ids=["default", "two levels", "three levels"])
def test_static_plan_matches_plan(g, opts):
    # two calls in a row on the static array, the second with a smaller input
    inputs = [(wl.rmat(12, 8, 0.57, 0.19, 0.19, 1),) * 2,
              (wl.rmat(11, 4, 0.57, 0.19, 0.19, 2), wl.rmat(11, 8, 0.57, 0.19, 0.19, 3))]
    for A, B in inputs:
        dA = g.DeviceCSR.from_host(A)
        dB = dA if B is A else g.DeviceCSR.from_host(B)
        ref = oracle.spgemm(A, B)
        rp0, col0, val0, info0 = _product(g, dA, dB, False, **opts)
        rp1, col1, val1, info1 = _product(g, dA, dB, True, **opts)
        assert np.array_equal(rp1, rp0) and np.array_equal(col1, col0)
        assert np.all(np.abs(val1 - val0) <= 2 * TOL * ref.bound)
        compare_full(rp1, col1, val1, ref)
        assert info1.n_heavy_rows == info0.n_heavy_rows and info1.c_nnz == info0.c_nnz
        assert 0 < info1.workspace_peak_bytes <= 128 << 20


def test_static_plans_coexist(g):
    # two static plans alive on one device take disjoint blocks of the array
    A = wl.rmat(12, 8, 0.57, 0.19, 0.19, 4)
    dA = g.DeviceCSR.from_host(A)
    ref = oracle.spgemm(A, A)
    with g.Plan(dA, dA, static_workspace=True, tau=300, dense_width_log2=7, chunks_max_log2=3) as p1, \
            g.Plan(dA, dA, static_workspace=True) as p2:
        rp1, _ = p1.symbolic()
        rp2, _ = p2.symbolic()
        c1, v1 = p1.numeric()
        c2, v2 = p2.numeric()
        torch.cuda.synchronize()
        for rp, c, v in ((rp1, c1, v1), (rp2, c2, v2)):
            compare_full(rp.cpu().numpy(), c.cpu().numpy(), v.cpu().numpy(), ref)


def test_static_plan_limits(g):
    # too many rows for the array: refused up front; a product whose heavy
    # path needs more than the array: OUT_OF_MEMORY, and the array is whole
    # again afterwards (a small product still runs)
    n = (128 << 20) // 41 + 1
    big = g.DeviceCSR(n, 4, torch.zeros(n + 1, dtype=torch.int64, device="cuda"),
                      torch.zeros(0, dtype=torch.int32, device="cuda"), torch.zeros(0, dtype=torch.float64,
                                                                                    device="cuda"))
    with pytest.raises(g.GmagnusError) as e:
        g.Plan(big, g.DeviceCSR(4, 4, torch.zeros(5, dtype=torch.int64, device="cuda"),
                                torch.zeros(0, dtype=torch.int32, device="cuda"),
                                torch.zeros(0, dtype=torch.float64, device="cuda")), static_workspace=True)
    assert e.value.status == 6 and "static workspace" in str(e.value)
    A = wl.rmat(16, 16, 0.57, 0.19, 0.19, 5)  # about 1.6e8 products, most of them in heavy rows
    dA = g.DeviceCSR.from_host(A)
    with pytest.raises(g.GmagnusError) as e:
        with g.Plan(dA, dA, static_workspace=True) as p:
            p.symbolic()
            p.numeric()
    assert e.value.status == 3
    B = wl.rmat(10, 8, 0.57, 0.19, 0.19, 6)
    dB = g.DeviceCSR.from_host(B)
    rp, col, val, _ = _product(g, dB, dB, True)
    compare_full(rp, col, val, oracle.spgemm(B, B))
    # allocator callbacks are refused
    with pytest.raises(g.GmagnusError) as e:
        g.Plan(dB, dB, static_workspace=True, alloc=g.ALLOC_FN(lambda n, s, c: None), free=g.FREE_FN(lambda p, s, c: None))
    assert e.value.status == 1
