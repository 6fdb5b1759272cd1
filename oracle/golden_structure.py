"""Writes the stored structure of C = A*A for the large workloads.

Test infrastructure: calls only the oracle (``oracle.row_counts``, the
symbolic phase of Section II-B by column marking) on inputs from the seeded
generators, and writes ``tests/golden/<config>_structure.txt``:

- the product count sum_i ip[i] and nnz(C);
- the sha256 of C's whole row-pointer array (n_rows + 1 little-endian int64,
  row_ptr[0] = 0);
- the sha256 of every block's row counts (n_rows / BLOCKS rows per block,
  little-endian int64), so that a mismatch names the rows it sits in.

Usage: python -m oracle.golden_structure [config ...]   (default: all four)
"""
from __future__ import annotations

import hashlib
import os
import sys
import time

import numpy as np

import oracle
import workloads as wl

BLOCKS = 128
DEFAULT = ("banded20", "er22", "rmat22", "rmat23")
GOLDEN = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "tests", "golden")


def structure_digests(counts: np.ndarray, blocks: int = BLOCKS):
    """(row_ptr sha256, [(row_begin, row_end, nnz, counts sha256)] per block) of per-row counts."""
    counts = np.ascontiguousarray(counts, dtype="<i8")
    rp = np.zeros(counts.size + 1, dtype="<i8")
    np.cumsum(counts, out=rp[1:])
    edges = [counts.size * b // blocks for b in range(blocks + 1)]
    per = []
    for b in range(blocks):
        s, e = edges[b], edges[b + 1]
        per.append((s, e, int(counts[s:e].sum()), hashlib.sha256(counts[s:e].tobytes()).hexdigest()))
    return hashlib.sha256(rp.tobytes()).hexdigest(), per


def _describe(cfg) -> str:
    return "%s %s, seed %d, values %s" % (cfg.kind, ", ".join(str(x) for x in cfg.params), cfg.seed, cfg.values)


def write(name: str) -> str:
    A = wl.CONFIGS[name].make()
    t = time.time()
    ip = oracle.row_products(A, A)
    counts = oracle.row_counts(A, A)
    secs = time.time() - t
    whole, per = structure_digests(counts)
    path = os.path.join(GOLDEN, "%s_structure.txt" % name)
    with open(path, "w") as f:
        f.write("# Structure of C = A*A for the %s workload (%s), from the oracle's symbolic\n" % (
            name, _describe(wl.CONFIGS[name])))
        f.write("# phase (distinct columns per row, Section II-B); written by oracle/golden_structure.py.\n")
        f.write("# row_ptr_sha256: sha256 of the n_rows + 1 row pointers as little-endian int64.\n")
        f.write("# block lines: row_begin row_end nnz sha256(row counts of the block, little-endian int64)\n")
        f.write("config %s\n" % name)
        f.write("n_rows %d\n" % A.n_rows)
        f.write("nnz_a %d\n" % A.nnz)
        f.write("products %d\n" % int(ip.sum()))
        f.write("nnz_c %d\n" % int(counts.sum()))
        f.write("row_ptr_sha256 %s\n" % whole)
        f.write("blocks %d\n" % len(per))
        for s, e, nz, h in per:
            f.write("block %d %d %d %s\n" % (s, e, nz, h))
    print("%s: nnz(C)=%d products=%d oracle %.1f s on %d threads -> %s" % (
        name, int(counts.sum()), int(ip.sum()), secs, oracle.threads(), path), flush=True)
    return path


def read(name: str) -> dict:
    """Parses tests/golden/<name>_structure.txt."""
    out = {"blocks": []}
    with open(os.path.join(GOLDEN, "%s_structure.txt" % name)) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            k, *v = line.split()
            if k == "block":
                out["blocks"].append((int(v[0]), int(v[1]), int(v[2]), v[3]))
            elif k in ("config", "row_ptr_sha256"):
                out[k] = v[0]
            elif k == "blocks":
                out["n_blocks"] = int(v[0])
            else:
                out[k] = int(v[0])
    return out


if __name__ == "__main__":
    for n in sys.argv[1:] or DEFAULT:
        write(n)
