"""MI355X (gfx950) SpGEMM C = A*B on CSR with the gMAGNUS heavy-row method.

The compute lives in libgmagnus.so (HIP kernels behind the C ABI declared in
include/gmagnus.h); :mod:`paper_2607_22866_amd.gmagnus` is its ctypes binding.
"""
from .gmagnus import (DeviceCSR, GmagnusError, Plan, get_params, load, release_cache, row_products, spgemm,
                      split_panels)

__all__ = ["DeviceCSR", "GmagnusError", "Plan", "get_params", "load", "release_cache", "row_products", "spgemm",
           "split_panels"]
