"""Thin ctypes binding of libgmagnus.so (include/gmagnus.h).

Argument marshalling only: torch tensors provide device memory and the HIP
stream; every step of the SpGEMM runs in the library's HIP kernels. There is
no fallback: if the library is missing or no GPU is present, calls raise.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgmagnus.so")

MAX_LEVELS = 8
K_NAMES = ["setup", "csc", "expand", "histogram", "multisplit", "chunk_symbolic", "chunk_numeric",
           "light_symbolic", "light_numeric", "rowptr"]
FLAG_TIMING = 1
FLAG_SERIAL_STREAMS = 2
FLAG_CONCURRENT_STREAMS = 128
FLAG_NO_WINDOW = 4
FLAG_PAPER_HISTOGRAM = 8
FLAG_PAPER_EXPANSION = 16
FLAG_SLICE_SPLIT = 32
FLAG_LEVEL_BY_LEVEL = 64
FLAG_KEEP_PATTERN = 256
PATH_NAMES = {0: "none", 1: "paper", 2: "slice_split", 3: "rows", 4: "rows_two_level"}

STATUS = {0: "SUCCESS", 1: "INVALID_VALUE", 2: "INVALID_CSR", 3: "OUT_OF_MEMORY", 4: "NOT_READY", 5: "HIP",
          6: "UNSUPPORTED"}


class GmagnusError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("%s: %s" % (STATUS.get(status, status), msg))
        self.status = status


class CsrDesc(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int64), ("n_cols", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("row_ptr", ctypes.c_void_p), ("col_idx", ctypes.c_void_p), ("val", ctypes.c_void_p)]


INDEX_TYPES = {torch.int32: 0, torch.int64: 1}
VALUE_TYPES = {torch.float64: 0, torch.float32: 1}


class MatrixDesc(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int64), ("n_cols", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("row_ptr", ctypes.c_void_p), ("col_idx", ctypes.c_void_p), ("val", ctypes.c_void_p),
                ("index_type", ctypes.c_int32), ("value_type", ctypes.c_int32)]


ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p)
FREE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p)


class Options(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_size_t), ("row_begin", ctypes.c_int64), ("row_end", ctypes.c_int64),
                ("lds_bytes", ctypes.c_int64), ("tau", ctypes.c_int64), ("dense_width_log2", ctypes.c_int32),
                ("chunks_max_log2", ctypes.c_int32), ("validate", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("alloc", ALLOC_FN), ("free", FREE_FN), ("alloc_ctx", ctypes.c_void_p),
                ("workspace_limit_bytes", ctypes.c_int64)]


class Params(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_int64), ("dense_width", ctypes.c_int64), ("chunks_required", ctypes.c_int64),
                ("chunks_max", ctypes.c_int64), ("min_group_elems", ctypes.c_int64), ("group_rows", ctypes.c_int64),
                ("n_levels", ctypes.c_int32), ("v_chunks", ctypes.c_int32 * MAX_LEVELS)]

    @property
    def levels(self):
        return [int(self.v_chunks[i]) for i in range(self.n_levels)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("params", Params), ("n_rows", ctypes.c_int64), ("n_heavy_rows", ctypes.c_int64),
                ("n_light_rows", ctypes.c_int64), ("products_total", ctypes.c_int64),
                ("products_heavy", ctypes.c_int64), ("n_slices", ctypes.c_int64), ("nnz_a_heavy", ctypes.c_int64),
                ("level_rows_in", ctypes.c_int64 * MAX_LEVELS), ("level_elems_in", ctypes.c_int64 * MAX_LEVELS),
                ("level_heavy_out", ctypes.c_int64 * MAX_LEVELS), ("levels_run", ctypes.c_int32),
                ("n_leaves_dense", ctypes.c_int64), ("n_leaves_hash", ctypes.c_int64),
                ("n_leaves_rank", ctypes.c_int64), ("c_nnz", ctypes.c_int64),
                ("c_nnz_heavy", ctypes.c_int64), ("check_flags", ctypes.c_int32),
                ("expansion_path", ctypes.c_int32), ("workspace_peak_bytes", ctypes.c_int64),
                ("index_type", ctypes.c_int32), ("value_type", ctypes.c_int32),
                ("kernel_ms", ctypes.c_double * len(K_NAMES)), ("kernel_launches", ctypes.c_int64 * len(K_NAMES)),
                ("kernel_bytes", ctypes.c_double * len(K_NAMES)), ("row_tau", ctypes.c_int64)]

    def to_dict(self) -> dict:
        d = {f: getattr(self, f) for f, _ in self._fields_ if f not in (
            "params", "level_rows_in", "level_elems_in", "level_heavy_out", "kernel_ms", "kernel_launches",
            "kernel_bytes")}
        p = self.params
        d["params"] = {"tau": p.tau, "dense_width": p.dense_width, "chunks_required": p.chunks_required,
                       "chunks_max": p.chunks_max, "v_chunks": p.levels}
        n = self.levels_run
        d["level_rows_in"] = list(self.level_rows_in[:n])
        d["level_elems_in"] = list(self.level_elems_in[:n])
        d["level_heavy_out"] = list(self.level_heavy_out[:n])
        d["kernels"] = {k: {"ms": self.kernel_ms[i], "launches": self.kernel_launches[i],
                            "bytes": self.kernel_bytes[i]} for i, k in enumerate(K_NAMES)}
        return d


EXPORTS = ["gmagnus_options_init", "gmagnus_get_params", "gmagnus_plan", "gmagnus_spgemm_symbolic",
           "gmagnus_spgemm_numeric", "gmagnus_plan_info", "gmagnus_plan_destroy", "gmagnus_row_products",
           "gmagnus_split_panels", "gmagnus_release_cache", "gmagnus_last_error", "gmagnus_status_string",
           "gmagnus_update_values", "gmagnus_expansion_path", "gmagnus_bandwidth_probe", "gmagnus_plan_static",
           "gmagnus_get_params_typed", "gmagnus_plan_typed", "gmagnus_spgemm_numeric_typed",
           "gmagnus_update_values_typed", "gmagnus_row_products_typed", "gmagnus_split_panels_typed"]

_lib = None


def load(path: str = LIB_PATH):
    """Loads libgmagnus.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libgmagnus.so not built (run python -m paper_2607_22866_amd.build)")
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    lib.gmagnus_options_init.argtypes = [ctypes.POINTER(Options)]
    lib.gmagnus_options_init.restype = None
    lib.gmagnus_get_params.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.POINTER(Options), ctypes.POINTER(Params)]
    lib.gmagnus_plan.argtypes = [ctypes.POINTER(P), ctypes.POINTER(CsrDesc), ctypes.POINTER(CsrDesc),
                                 ctypes.POINTER(Options), P]
    lib.gmagnus_plan_static.argtypes = lib.gmagnus_plan.argtypes
    M = ctypes.POINTER(MatrixDesc)
    lib.gmagnus_get_params_typed.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                             ctypes.POINTER(Options), ctypes.POINTER(Params)]
    lib.gmagnus_plan_typed.argtypes = [ctypes.POINTER(P), M, M, ctypes.POINTER(Options), P]
    lib.gmagnus_spgemm_numeric_typed.argtypes = [P, P, P, P]
    lib.gmagnus_update_values_typed.argtypes = [P, P, P]
    lib.gmagnus_row_products_typed.argtypes = [M, M, P, P]
    lib.gmagnus_split_panels_typed.argtypes = [M, M, ctypes.c_int64, P, ctypes.c_int64, ctypes.POINTER(ctypes.c_int64),
                                               P]
    lib.gmagnus_spgemm_symbolic.argtypes = [P, P, ctypes.POINTER(ctypes.c_int64)]
    lib.gmagnus_spgemm_numeric.argtypes = [P, P, P, P]
    lib.gmagnus_update_values.argtypes = [P, P, P]
    lib.gmagnus_plan_info.argtypes = [P, ctypes.POINTER(PlanInfo)]
    lib.gmagnus_plan_destroy.argtypes = [P]
    lib.gmagnus_plan_destroy.restype = None
    lib.gmagnus_row_products.argtypes = [ctypes.POINTER(CsrDesc), ctypes.POINTER(CsrDesc), P, P]
    lib.gmagnus_split_panels.argtypes = [ctypes.POINTER(CsrDesc), ctypes.POINTER(CsrDesc), ctypes.c_int64, P,
                                         ctypes.c_int64, ctypes.POINTER(ctypes.c_int64), P]
    lib.gmagnus_expansion_path.argtypes = [ctypes.POINTER(Params), ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                           ctypes.c_int32]
    lib.gmagnus_expansion_path.restype = ctypes.c_int32
    lib.gmagnus_bandwidth_probe.argtypes = [ctypes.c_int32, P, P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, P,
                                            ctypes.POINTER(ctypes.c_double)]
    lib.gmagnus_bandwidth_probe.restype = ctypes.c_int
    lib.gmagnus_release_cache.argtypes = []
    lib.gmagnus_release_cache.restype = None
    lib.gmagnus_last_error.restype = ctypes.c_char_p
    lib.gmagnus_status_string.argtypes = [ctypes.c_int]
    lib.gmagnus_status_string.restype = ctypes.c_char_p
    for f in ("gmagnus_get_params", "gmagnus_plan", "gmagnus_plan_static", "gmagnus_spgemm_symbolic", "gmagnus_spgemm_numeric",
              "gmagnus_update_values", "gmagnus_plan_info", "gmagnus_row_products", "gmagnus_split_panels",
              "gmagnus_get_params_typed", "gmagnus_plan_typed", "gmagnus_spgemm_numeric_typed",
              "gmagnus_update_values_typed", "gmagnus_row_products_typed", "gmagnus_split_panels_typed"):
        getattr(lib, f).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(st: int):
    if st != 0:
        raise GmagnusError(st, load().gmagnus_last_error().decode())


def make_options(**kw) -> Options:
    o = Options()
    load().gmagnus_options_init(ctypes.byref(o))
    for k, v in kw.items():
        if v is None:
            continue
        if not hasattr(o, k):
            raise TypeError("unknown option %r" % k)
        setattr(o, k, v)
    return o


def get_params(c_m: int, lds_bytes: int = 163840, index_dtype=torch.int32, value_dtype=torch.float64,
               **overrides) -> Params:
    """Host-only parameter selection of the library (no GPU needed) for the
    given column-index and value types."""
    p = Params()
    o = make_options(**overrides)
    _check(load().gmagnus_get_params_typed(c_m, lds_bytes, INDEX_TYPES[index_dtype], VALUE_TYPES[value_dtype],
                                           ctypes.byref(o), ctypes.byref(p)))
    return p


def expansion_path(params: Params, n_heavy: int, products_heavy: int, b_nnz: int, flags: int = 0) -> str:
    """Host-only: the expansion order a plan with these parameters takes (a PATH_NAMES value)."""
    return PATH_NAMES[int(load().gmagnus_expansion_path(ctypes.byref(params), n_heavy, products_heavy, b_nnz,
                                                        flags))]


def _require_device(t: torch.Tensor, device: torch.device, name: str):
    """The library reads and writes device memory only: a host tensor's pointer
    handed to a kernel would fault the GPU, so it is refused here."""
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError("%s must be a CUDA tensor" % name)
    if t.device != device:
        raise ValueError("%s is on %s, the plan's matrices on %s" % (name, t.device, device))


@dataclass
class DeviceCSR:
    """CSR on the GPU (torch tensors): int64 row_ptr, int32 or int64 col,
    float64 or float32 val."""

    n_rows: int
    n_cols: int
    row_ptr: torch.Tensor
    col: torch.Tensor
    val: torch.Tensor

    @property
    def nnz(self) -> int:
        return int(self.col.numel())

    @staticmethod
    def from_host(m, device="cuda", index_dtype=torch.int32, value_dtype=torch.float64) -> "DeviceCSR":
        """Copies a host CSR (numpy or torch arrays) to the device, converting
        its columns and values to the given types."""
        rp = torch.as_tensor(m.row_ptr, dtype=torch.int64).to(device)
        col = torch.as_tensor(m.col).to(index_dtype).to(device)
        val = torch.as_tensor(m.val).to(value_dtype).to(device)
        return DeviceCSR(int(m.n_rows), int(m.n_cols), rp, col, val)

    @property
    def index_dtype(self):
        return self.col.dtype

    @property
    def value_dtype(self):
        return self.val.dtype

    def _check_arrays(self):
        if (not all(t.is_cuda and t.is_contiguous() for t in (self.row_ptr, self.col, self.val))
                or self.row_ptr.dtype != torch.int64 or self.col.dtype not in INDEX_TYPES
                or self.val.dtype not in VALUE_TYPES):
            raise ValueError("DeviceCSR arrays must be contiguous CUDA tensors: int64 row_ptr, int32/int64 col, "
                             "float64/float32 val")

    def desc(self) -> CsrDesc:
        """The int32 / fp64 descriptor of gmagnus_csr_t."""
        self._check_arrays()
        if self.col.dtype != torch.int32 or self.val.dtype != torch.float64:
            raise ValueError("gmagnus_csr_t takes int32 columns and float64 values")
        return CsrDesc(self.n_rows, self.n_cols, self.nnz, self.row_ptr.data_ptr(),
                       self.col.data_ptr() if self.nnz else None, self.val.data_ptr() if self.nnz else None)

    def mdesc(self) -> MatrixDesc:
        """The typed descriptor of gmagnus_matrix_t."""
        self._check_arrays()
        return MatrixDesc(self.n_rows, self.n_cols, self.nnz, self.row_ptr.data_ptr(),
                          self.col.data_ptr() if self.nnz else None, self.val.data_ptr() if self.nnz else None,
                          INDEX_TYPES[self.col.dtype], VALUE_TYPES[self.val.dtype])

    def to_host(self):
        return self.row_ptr.cpu().numpy(), self.col.cpu().numpy(), self.val.cpu().numpy()


def _stream(stream) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


class Plan:
    """One row panel of C = A*B: setup on construction, then symbolic and numeric.
    static_workspace=True builds it with gmagnus_plan_static (no device
    allocation by the library: its workspace is a static device array)."""

    def __init__(self, A: DeviceCSR, B: DeviceCSR, stream=None, static_workspace: bool = False, **options):
        self._lib = load()
        self.A, self.B = A, B  # borrowed by the library until close()
        self._opts = make_options(**options)
        self._stream = stream
        self._h = ctypes.c_void_p()
        if static_workspace:
            self._da, self._db = A.desc(), B.desc()
            make = self._lib.gmagnus_plan_static
        else:
            self._da, self._db = A.mdesc(), B.mdesc()
            make = self._lib.gmagnus_plan_typed
        _check(make(ctypes.byref(self._h), ctypes.byref(self._da), ctypes.byref(self._db), ctypes.byref(self._opts),
                    _stream(stream)))
        rb = self._opts.row_begin
        re = self._opts.row_end if self._opts.row_end > 0 else A.n_rows
        self.n_rows = re - rb
        self.row_ptr: Optional[torch.Tensor] = None
        self.nnz = None

    def symbolic(self):
        """Returns (row_ptr of the panel on the device, nnz)."""
        rp = torch.empty(self.n_rows + 1, dtype=torch.int64, device=self.A.row_ptr.device)
        nnz = ctypes.c_int64()
        _check(self._lib.gmagnus_spgemm_symbolic(self._h, rp.data_ptr(), ctypes.byref(nnz)))
        self.row_ptr, self.nnz = rp, int(nnz.value)
        return rp, self.nnz

    def numeric(self, col: Optional[torch.Tensor] = None, val: Optional[torch.Tensor] = None):
        """Fills (and returns) C's column and value arrays for the panel."""
        dev = self.A.row_ptr.device
        if col is None:
            col = torch.empty(self.nnz, dtype=self.A.col.dtype, device=dev)
        if val is None:
            val = torch.empty(self.nnz, dtype=self.A.val.dtype, device=dev)
        for t, dt, name in ((col, self.A.col.dtype, "col"), (val, self.A.val.dtype, "val")):
            _require_device(t, dev, name)
            if t.dtype != dt or not t.is_contiguous():
                raise ValueError("%s must be a contiguous %s array" % (name, dt))
        if col.numel() < self.nnz or val.numel() < self.nnz:
            raise ValueError("output arrays smaller than nnz")
        _check(self._lib.gmagnus_spgemm_numeric_typed(self._h, self.row_ptr.data_ptr(),
                                                col.data_ptr() if self.nnz else None,
                                                val.data_ptr() if self.nnz else None))
        return col, val

    def update_values(self, a_val: torch.Tensor, b_val: Optional[torch.Tensor] = None):
        """New values of A and B (float64 device arrays in their CSR order) on
        the same patterns; needs flags=FLAG_KEEP_PATTERN at construction. The next
        numeric() writes C for these values. b_val defaults to a_val when the
        plan's A and B are one matrix."""
        if b_val is None:
            if self.B is not self.A:
                raise ValueError("b_val is required when A and B differ")
            b_val = a_val
        for t, m, name in ((a_val, self.A, "a_val"), (b_val, self.B, "b_val")):
            _require_device(t, self.A.row_ptr.device, name)
            if t.dtype != m.val.dtype or not t.is_contiguous() or t.numel() < m.nnz:
                raise ValueError("%s must be a contiguous %s array of at least nnz entries" % (name, m.val.dtype))
        self._vals = (a_val, b_val)  # borrowed by the library until the next numeric phase ends
        _check(self._lib.gmagnus_update_values_typed(self._h, a_val.data_ptr() if self.A.nnz else None,
                                               b_val.data_ptr() if self.B.nnz else None))

    def info(self) -> PlanInfo:
        out = PlanInfo()
        _check(self._lib.gmagnus_plan_info(self._h, ctypes.byref(out)))
        return out

    def close(self):
        if self._h:
            self._lib.gmagnus_plan_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def spgemm(A: DeviceCSR, B: DeviceCSR, stream=None, **options):
    """C = A*B for the rows selected by options (default all): (row_ptr, col, val) on the device."""
    with Plan(A, B, stream=stream, **options) as p:
        rp, _ = p.symbolic()
        col, val = p.numeric()
        return rp, col, val


def row_products(A: DeviceCSR, B: DeviceCSR, stream=None) -> torch.Tensor:
    ip = torch.empty(A.n_rows, dtype=torch.int64, device=A.row_ptr.device)
    da, db = A.mdesc(), B.mdesc()
    _check(load().gmagnus_row_products_typed(ctypes.byref(da), ctypes.byref(db), ip.data_ptr() if A.n_rows else None,
                                       _stream(stream)))
    return ip


def split_panels(A: DeviceCSR, B: DeviceCSR, max_products: int, max_panels: int = 1 << 16, stream=None):
    bounds = (ctypes.c_int64 * (max_panels + 1))()
    n = ctypes.c_int64()
    da, db = A.mdesc(), B.mdesc()
    _check(load().gmagnus_split_panels_typed(ctypes.byref(da), ctypes.byref(db), max_products, bounds, max_panels,
                                       ctypes.byref(n), _stream(stream)))
    return [int(bounds[i]) for i in range(n.value + 1)]


PROBE_KINDS = {"read": 0, "read_nt": 1, "write": 2, "write_nt": 3, "copy": 4, "gather": 5}
GATHER_PROBE_BYTES = 4 << 30  # bytes one gather probe run reads


def bandwidth_probe(kind: str, nbytes: int = 4 << 30, reps: int = 5, grid: int = 0, stream=None) -> float:
    """Bandwidth of one probe kernel in GB/s (bytes moved / time; a copy moves
    its bytes twice; "gather" reads GATHER_PROBE_BYTES as random lines of a
    working set of nbytes bytes)."""
    k = PROBE_KINDS[kind]
    src = torch.ones(nbytes // 8, dtype=torch.float64, device="cuda")
    dst = torch.empty_like(src) if kind not in ("read", "read_nt", "gather") else torch.zeros(
        1, dtype=torch.float64, device="cuda")
    ms = ctypes.c_double()
    _check(load().gmagnus_bandwidth_probe(k, dst.data_ptr(), src.data_ptr(), nbytes, grid, reps, _stream(stream),
                                          ctypes.byref(ms)))
    del src, dst
    moved = 2 * nbytes if kind == "copy" else GATHER_PROBE_BYTES if kind == "gather" else nbytes
    return moved / (ms.value / 1000.0) / 1e9


def release_cache():
    load().gmagnus_release_cache()
