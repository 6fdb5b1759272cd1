"""CPU-side checks of the C ABI: the library loads, exports every declared
symbol, its host-only planner matches the paper's printed chunk counts, and
argument validation fails with status codes before touching a device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gmagnus.h")

gm = pytest.importorskip("paper_2607_22866_amd.gmagnus")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(gm.LIB_PATH):
        from paper_2607_22866_amd import build

        build.build()
    return gm.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gmagnus_\w+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(gm.EXPORTS) == names


def test_struct_sizes_match_header(lib):
    # the options struct carries its own size; a mismatch is rejected
    o = gm.make_options()
    assert o.struct_size == ctypes.sizeof(gm.Options)
    p = gm.Params()
    o.struct_size = 8
    assert lib.gmagnus_get_params(4096, 163840, ctypes.byref(o), ctypes.byref(p)) == 1


def _golden():
    rows = []
    with open(os.path.join(ROOT, "tests", "golden", "num_chunks.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([x.strip() for x in line.split("|")])
    return rows


def _fmt(p):
    lv = p.levels
    if len(lv) <= 1:
        return str(p.chunks_required)
    return "%d: %s" % (p.chunks_required, ", ".join(map(str, lv)))


def test_library_planner_reproduces_printed_chunk_counts(lib):
    n = 0
    for name, cm, pvc, h200 in _golden():
        for s_lm, printed in ((131072, pvc), (233472, h200)):
            if printed == "N/A":
                continue
            assert _fmt(gm.get_params(int(cm), s_lm)) == printed, (name, s_lm)
            n += 1
    assert n == 51


def test_library_planner_matches_oracle_planner(lib):
    from oracle.params import get_magnus_params

    for s_lm in (65536, 131072, 163840, 233472):
        for cm in (1, 100, 4096, 8192, 8193, 65536, 1 << 20, (1 << 22) + 3, 1 << 23, 1 << 26, 2_000_000_000):
            a = gm.get_params(cm, s_lm)
            b = get_magnus_params(cm, s_lm)
            assert (a.dense_width, a.chunks_required, a.chunks_max) == (b.dense_width, b.chunks_required,
                                                                        b.chunks_max), (cm, s_lm)
            assert a.levels == b.v_chunks, (cm, s_lm)
            assert a.tau == min(b.tau, 6912)  # the library clamps tau to its light accumulators' capacity


def test_planner_mi355x_defaults(lib):
    p = gm.get_params(1 << 22, 163840)
    assert (p.tau, p.dense_width, p.chunks_max, p.levels) == (6826, 8192, 32, [32, 16])
    assert gm.get_params(1 << 23).levels == [32, 32]
    assert gm.get_params(4096).levels == []
    # overrides force any depth on a small column count
    assert gm.get_params(4096, tau=200, dense_width_log2=6, chunks_max_log2=2).levels == [4, 4, 4]
    assert gm.get_params(4096, dense_width_log2=8, chunks_max_log2=4).levels == [16]
    assert gm.get_params(4096, dense_width_log2=7, chunks_max_log2=3).levels == [8, 4]


def test_planner_rejects_bad_arguments(lib):
    for cm, lds, kw in ((0, 163840, {}), (1 << 31, 163840, {}), (4096, 100, {}), (4096, 163840,
                                                                                  {"dense_width_log2": 14})):
        with pytest.raises(gm.GmagnusError) as e:
            gm.get_params(cm, lds, **kw)
        assert e.value.status == 1


def _desc(n_rows, n_cols, nnz=0, ptr=0x1000):
    return gm.CsrDesc(n_rows, n_cols, nnz, ptr, ptr if nnz else None, ptr if nnz else None)


def test_plan_argument_validation_without_device(lib):
    h = ctypes.c_void_p()
    a, b = _desc(4, 5), _desc(6, 3)
    # NULL output
    assert lib.gmagnus_plan(None, ctypes.byref(a), ctypes.byref(b), None, None) == 1
    # NULL operand
    assert lib.gmagnus_plan(ctypes.byref(h), None, ctypes.byref(b), None, None) == 1
    assert not h.value
    # inner dimensions differ
    assert lib.gmagnus_plan(ctypes.byref(h), ctypes.byref(a), ctypes.byref(b), None, None) == 1
    assert b"A.n_cols" in lib.gmagnus_last_error()
    # too many columns
    big = _desc(4, 1 << 31)
    assert lib.gmagnus_plan(ctypes.byref(h), ctypes.byref(_desc(4, 4)), ctypes.byref(_desc(4, 1 << 31)), None,
                            None) == 6
    # option struct of another size
    o = gm.make_options()
    o.struct_size = 4
    b2 = _desc(5, 3)
    assert lib.gmagnus_plan(ctypes.byref(h), ctypes.byref(a), ctypes.byref(b2), ctypes.byref(o), None) == 1
    # NULL plan handles
    nnz = ctypes.c_int64()
    assert lib.gmagnus_spgemm_symbolic(None, None, ctypes.byref(nnz)) == 1
    assert lib.gmagnus_spgemm_numeric(None, None, None, None) == 1
    assert lib.gmagnus_plan_info(None, None) == 1
    lib.gmagnus_plan_destroy(None)
    del big


def test_status_strings(lib):
    for code, name in gm.STATUS.items():
        assert lib.gmagnus_status_string(code).decode() == "GMAGNUS_" + ("SUCCESS" if code == 0 else "ERROR_" + name)


def test_expansion_path_predicate(lib):
    # the routing of the heavy rows (host-only): paper order without a level or
    # when asked; row order when its 32-bit offsets fit; both levels fused only
    # for two-level hierarchies whose B can be indexed in 32 bits
    p2 = gm.get_params(1 << 22)  # [32, 16]
    p1 = gm.get_params(1 << 17)  # one level
    p0 = gm.get_params(4096)     # no level
    path = gm.expansion_path
    assert path(p2, 0, 0, 100) == "none"
    assert path(p0, 10, 10_000, 100) == "paper"
    assert path(p2, 10, 10_000, 100, gm.FLAG_PAPER_EXPANSION) == "paper"
    assert path(p2, 10, 10_000, 100, gm.FLAG_PAPER_HISTOGRAM) == "paper"
    assert path(p2, 10, 10_000, 100, gm.FLAG_SLICE_SPLIT) == "slice_split"
    assert path(p2, 10, 1 << 32, 100) == "slice_split"          # offsets past 32 bits
    assert path(p2, 10, (1 << 32) - 1, 100) == "rows_two_level"
    assert path(p2, 10, 10_000, 100) == "rows_two_level"
    assert path(p2, 10, 10_000, 100, gm.FLAG_LEVEL_BY_LEVEL) == "rows"
    assert path(p2, 10, 10_000, (1 << 31) - 1) == "rows_two_level"
    assert path(p2, 10, 10_000, 1 << 31) == "rows"               # B.nnz past 32-bit fine boundaries
    assert path(p1, 10, 10_000, 100) == "rows"
    assert path(gm.get_params(1 << 23), 10, 10_000, 100) == "rows_two_level"
    assert path(gm.get_params(4096, tau=200, dense_width_log2=6, chunks_max_log2=2), 10, 10_000, 100) == "rows"


def test_binding_refuses_host_tensors(lib):
    # a host tensor's pointer in a kernel would fault the GPU: the binding
    # refuses it before any library call (the plan below has no library)
    import types

    import torch

    p = gm.Plan.__new__(gm.Plan)
    p._lib = None  # any library call would raise AttributeError, not ValueError
    p._h = ctypes.c_void_p()
    m = types.SimpleNamespace(row_ptr=torch.zeros(3, dtype=torch.int64), col=torch.zeros(2, dtype=torch.int32),
                              val=torch.zeros(2, dtype=torch.float64), nnz=2)
    p.A = p.B = m
    p.nnz = 2
    p.row_ptr = torch.zeros(3, dtype=torch.int64)
    col, val = torch.zeros(2, dtype=torch.int32), torch.zeros(2, dtype=torch.float64)
    with pytest.raises(ValueError, match="CUDA tensor"):
        p.numeric(col, val)
    with pytest.raises(ValueError, match="CUDA tensor"):
        p.update_values(val, val)


def test_probe_argument_validation(lib):
    ms = ctypes.c_double()
    assert lib.gmagnus_bandwidth_probe(9, 0x1000, 0x1000, 1 << 20, 0, 1, None, ctypes.byref(ms)) == 1
    assert lib.gmagnus_bandwidth_probe(4, 0x1000, 0x1000, 17, 0, 1, None, ctypes.byref(ms)) == 1
    assert lib.gmagnus_bandwidth_probe(4, 0x1000, None, 1 << 20, 0, 1, None, ctypes.byref(ms)) == 1
    assert lib.gmagnus_bandwidth_probe(4, 0x1008, 0x1000, 1 << 20, 0, 1, None, ctypes.byref(ms)) == 1
    assert lib.gmagnus_bandwidth_probe(4, 0x1000, 0x1000, 1 << 20, 0, 0, None, ctypes.byref(ms)) == 1


TYPE_SIZES = [("int32", "float64", 4, 8), ("int32", "float32", 4, 4), ("int64", "float64", 8, 8),
              ("int64", "float32", 8, 4)]


@pytest.mark.parametrize("idt,vdt,s_col,s_val", TYPE_SIZES)
def test_typed_planner_matches_oracle_planner(lib, idt, vdt, s_col, s_val):
    # tau, W and the chunk limits from the type sizes (Section III-D), with the
    # library's caps on tau (light-row capacity) and W (dense accumulator)
    import torch

    from oracle.params import get_magnus_params

    it, vt = getattr(torch, idt), getattr(torch, vdt)
    for s_lm in (65536, 131072, 163840, 233472):
        for cm in (1, 100, 4096, 8193, 65536, 1 << 20, (1 << 22) + 3, 1 << 23, 2_000_000_000):
            a = gm.get_params(cm, s_lm, it, vt)
            b = get_magnus_params(cm, s_lm, s_col=s_col, s_val=s_val, dense_width_max=8192, tau_max=6912)
            assert (a.tau, a.dense_width, a.chunks_required, a.chunks_max) == (b.tau, b.dense_width,
                                                                               b.chunks_required, b.chunks_max)
            assert a.levels == b.v_chunks, (cm, s_lm)


def test_typed_planner_values_at_160kb(lib):
    import torch

    p = gm.get_params(1 << 22, 163840, torch.int64, torch.float64)
    assert (p.tau, p.dense_width, p.chunks_max, p.levels) == (5120, 8192, 32, [32, 16])
    p = gm.get_params(1 << 22, 163840, torch.int32, torch.float32)  # tau 10240 and W 16384 derived, then capped
    assert (p.tau, p.dense_width, p.chunks_max, p.levels) == (6912, 8192, 64, [64, 8])
    p = gm.get_params(1 << 22, 163840, torch.int64, torch.float32)
    assert (p.tau, p.dense_width, p.chunks_max, p.levels) == (6826, 8192, 32, [32, 16])
    # int64 columns reach 2^35 columns of C; int32 stays below 2^31
    assert gm.get_params(1 << 35, 163840, torch.int64, torch.float64).levels == [32, 32, 32, 32, 4]
    for cm, it in (((1 << 35) + 1, torch.int64), (1 << 31, torch.int32)):
        with pytest.raises(gm.GmagnusError) as e:
            gm.get_params(cm, 163840, it, torch.float64)
        assert e.value.status == 1


def test_typed_plan_validation_without_device(lib):
    h = ctypes.c_void_p()

    def md(n_rows, n_cols, it=0, vt=0):
        return gm.MatrixDesc(n_rows, n_cols, 0, 0x1000, None, None, it, vt)
    # mismatched types
    assert lib.gmagnus_plan_typed(ctypes.byref(h), ctypes.byref(md(4, 5, 0, 0)), ctypes.byref(md(5, 3, 1, 0)), None,
                                  None) == 1
    assert lib.gmagnus_plan_typed(ctypes.byref(h), ctypes.byref(md(4, 5, 0, 0)), ctypes.byref(md(5, 3, 0, 1)), None,
                                  None) == 1
    # unknown types
    assert lib.gmagnus_plan_typed(ctypes.byref(h), ctypes.byref(md(4, 5, 2, 0)), ctypes.byref(md(5, 3, 2, 0)), None,
                                  None) == 1
    # int64 columns allow B (C) up to 2^35 columns, never A
    assert lib.gmagnus_plan_typed(ctypes.byref(h), ctypes.byref(md(4, 1 << 31, 1)), ctypes.byref(md(1 << 31, 3, 1)),
                                  None, None) == 6
    assert lib.gmagnus_plan_typed(ctypes.byref(h), ctypes.byref(md(4, 5, 1)), ctypes.byref(md(5, (1 << 35) + 1, 1)),
                                  None, None) == 6
    assert not h.value
