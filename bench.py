"""Benchmark: SpGEMM C = A*A (C = A*B for the R-MAT pairs) on one MI355X through the C ABI.

One step = the whole product for the workload: row-panel split by product
counts, then per panel the setup (row products, light/heavy split), the
symbolic phase (heavy expansion, hierarchical multisplit, final-chunk and
light-row counts, C row pointers) and the numeric phase (C columns and
values). Inputs are resident in HBM before timing starts; each panel of C is
written to HBM (panels reuse one allocation when C does not fit at once).

Prints one JSON line (see the repository's benchmark contract). The
roofline object is for the single kernel (one launch per panel) with the
largest device time: its algorithmic bytes per launch over its average
launch time, measured with HIP events on the stream it runs on. Its
"traffic" is the HBM bytes per launch from the committed rocprofv3 counter
summary (FETCH_SIZE + WRITE_SIZE scaled by a copy kernel's reading), or null
when there is none or the kernel's sources changed since it was taken. The
oracle is timed on a bounded sample of rows for the CPU baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "SpGEMM GFLOP/s (2×intermediate products/s) + achieved HBM GB/s, C=A·A"
WORKLOADS = {
    "rmat12": "R-MAT scale 12 (4096x4096), edge factor 8, (a,b,c,d)=(0.57,0.19,0.19,0.05), fp64 U(0,1), C=A*A",
    "banded20": "Banded 2^20 x 2^20, 27 nnz/row at offsets -13..+13, fp64 U(-1,1), C=A*A",
    "er22": "Erdos-Renyi 2^22 x 2^22, 16 nnz/row uniform without replacement, fp64 U(-1,1), C=A*A",
    "rmat22": "R-MAT scale 22 (2^22 x 2^22), edge factor 16, (a,b,c,d)=(0.57,0.19,0.19,0.05), fp64 U(0,1), C=A*A",
    "rmat23": "R-MAT scale 23 (2^23 x 2^23), edge factor 8, (a,b,c,d)=(0.60,0.17,0.17,0.06), fp64 U(0,1), C=A*A",
}
# A*B pairs (two R-MAT matrices of one scale, different edge factors); not the headline workload.
PAIR_WORKLOADS = {
    "rmat20_a32_b8": "R-MAT scale 20, A edge factor 32 times B edge factor 8, (a,b,c,d)=(0.57,0.19,0.19,0.05), "
                     "fp64 U(0,1), C=A*B",
    "rmat20_a64_b16": "R-MAT scale 20, A edge factor 64 times B edge factor 16, (a,b,c,d)=(0.57,0.19,0.19,0.05), "
                      "fp64 U(0,1), C=A*B",
}
HEAVY_KERNELS = ["expand", "histogram", "multisplit", "chunk_symbolic", "chunk_numeric"]
# Timing classes that are exactly one kernel launch per panel: the roofline is
# reported for the one of these with the largest device time.
SINGLE_KERNEL_CLASSES = {"expand": "k_expand_rows2", "multisplit": "k_multisplit"}
# Sources a kernel's counter summary depends on (traffic is dropped when they change).
KERNEL_SOURCES = {"k_expand_rows2": ["paper_2607_22866_amd/csrc/rowsplit.hip", "paper_2607_22866_amd/csrc/common.hpp"],
                  "k_expand_rows": ["paper_2607_22866_amd/csrc/rowsplit.hip", "paper_2607_22866_amd/csrc/common.hpp"],
                  "k_expand_split": ["paper_2607_22866_amd/csrc/expand.hip", "paper_2607_22866_amd/csrc/common.hpp"],
                  "k_expand": ["paper_2607_22866_amd/csrc/expand.hip", "paper_2607_22866_amd/csrc/common.hpp"],
                  "k_multisplit": ["paper_2607_22866_amd/csrc/multisplit.hip",
                                   "paper_2607_22866_amd/csrc/common.hpp"]}
TRAFFIC_FILES = {"k_expand_rows2": "profiles/expand_rows2_rmat22_traffic.md",
                 "k_expand_rows": "profiles/expand_rows_rmat22_traffic.md",
                 "k_expand_split": "profiles/expand_split_rmat22_traffic.md",
                 "k_multisplit": "profiles/multisplit_rmat22_traffic.md"}


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def run_step(g, dA, dB, bounds, timing, acc, c_bufs, extra_flags=0, tau=0):
    """One full product; returns (products, nnz(C))."""
    import torch

    products = 0
    nnz = 0
    flags = (g.FLAG_TIMING if timing else 0) | extra_flags
    for a, b in zip(bounds[:-1], bounds[1:]):
        with g.Plan(dA, dB, row_begin=a, row_end=b, flags=flags, tau=tau) as p:
            rp, n = p.symbolic()
            if c_bufs[0] is None or c_bufs[0].numel() < n:
                c_bufs[0] = c_bufs[1] = None
                c_bufs[0] = torch.empty(max(n, 1), dtype=torch.int32, device="cuda")
                c_bufs[1] = torch.empty(max(n, 1), dtype=torch.float64, device="cuda")
            p.numeric(c_bufs[0], c_bufs[1])
            info = p.info() if timing else None
        nnz += n
        if info is not None:
            if info.check_flags != 0:
                raise RuntimeError("panel [%d, %d): the library's consistency flags are %d (a kernel's output "
                                   "disagreed with the symbolic phase); the step's result is wrong" % (
                                       a, b, info.check_flags))
            products += info.products_total
            acc["_heavy"] = acc.get("_heavy", 0) + info.products_heavy
            acc.setdefault("_levels", set()).add(info.params.n_levels)
            for i, k in enumerate(g.K_NAMES):
                acc.setdefault(k, [0.0, 0, 0.0])
                acc[k][0] += info.kernel_ms[i]
                acc[k][1] += info.kernel_launches[i]
                acc[k][2] += info.kernel_bytes[i]
    return products, nnz


def reuse_pass(g, dA, dB, bounds, c_bufs, extra_flags=0, tau=0):
    """Pattern reuse, panel by panel: the full product (plan, symbolic,
    numeric) on a plan that keeps its pattern, then new values of A and B
    (gmagnus_update_values) and numeric again. Returns the summed seconds of
    the full products and of the values-only re-runs."""
    import torch

    va = (dA.val * 0.5 + 0.25).contiguous()
    vb = va if dB is dA else (dB.val * 0.5 + 0.25).contiguous()
    t_full = t_vals = 0.0
    for a, b in zip(bounds[:-1], bounds[1:]):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        with g.Plan(dA, dB, row_begin=a, row_end=b, flags=g.FLAG_KEEP_PATTERN | extra_flags, tau=tau) as p:
            rp, n = p.symbolic()
            if c_bufs[0] is None or c_bufs[0].numel() < n:
                c_bufs[0] = c_bufs[1] = None
                c_bufs[0] = torch.empty(max(n, 1), dtype=torch.int32, device="cuda")
                c_bufs[1] = torch.empty(max(n, 1), dtype=torch.float64, device="cuda")
            p.numeric(c_bufs[0], c_bufs[1])
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            p.update_values(va, vb)
            p.numeric(c_bufs[0], c_bufs[1])
            torch.cuda.synchronize()
            t2 = time.perf_counter()
        t_full += t1 - t0
        t_vals += t2 - t1
    return t_full, t_vals


def measured_peaks(g):
    """Streaming bandwidths of the library's probe kernels (4 GiB, 5 runs
    each): the measured peaks the paper divides by in its speed-of-light
    comparison (copy), with read-only and write-only ceilings beside it."""
    import torch

    out = {k: g.bandwidth_probe(k) for k in ("read", "read_nt", "write", "write_nt", "copy")}
    torch.cuda.empty_cache()
    return out


def cache_probe(g):
    """Rate of random 128-byte line reads (the expansion's B-row gathers)
    against the size of the working set they fall in, GB/s: sizes the L2s
    (4 MB per XCD) hold run far above HBM, larger ones at the memory side's
    rate."""
    import torch

    out = {}
    for log2 in range(21, 33):
        out["%d MiB" % (1 << (log2 - 20))] = g.bandwidth_probe("gather", nbytes=1 << log2, reps=3)
    torch.cuda.empty_cache()
    return out


def cpu_description():
    """Model name of the host CPU and the logical CPUs this process may use."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        logical = len(os.sched_getaffinity(0))
    except AttributeError:
        logical = os.cpu_count()
    return model, logical


def source_hash(kernel):
    """Hash of the kernel's sources with comments and whitespace removed (so a
    comment edit does not invalidate its counter summary)."""
    import hashlib
    import re

    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, f)) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic(kernel, config):
    """HBM bytes per launch from the committed counter summary of this kernel
    (FETCH_SIZE + WRITE_SIZE, scaled by the copy-kernel calibration), or None
    when there is none for this workload or the kernel changed since."""
    path = os.path.join(ROOT, TRAFFIC_FILES.get(kernel, ""))
    if not os.path.isfile(path):
        return None
    vals = {}
    with open(path) as fh:
        for line in fh:
            if line.startswith("traffic:"):
                k, _, v = line[len("traffic:"):].strip().partition("=")
                vals[k.strip()] = v.strip()
    if vals.get("source_hash") != source_hash(kernel) or vals.get("config") != config:
        return None
    return float(vals["bytes_per_launch"])


def cpu_baseline(A, B, ip, budget_products, seed=0):
    """Times the oracle on a random sample of rows (about budget_products products)."""
    import numpy as np

    import oracle

    rng = np.random.default_rng(seed)
    order = rng.permutation(A.n_rows)
    csum = np.cumsum(ip[order])
    k = int(np.searchsorted(csum, budget_products)) + 1
    rows = np.sort(order[:k])
    sample_products = int(ip[rows].sum())
    t0 = time.perf_counter()
    oracle.spgemm(A, B, rows=rows)
    dt = time.perf_counter() - t0
    model, logical = cpu_description()
    return {
        "value": 2.0 * sample_products / dt / 1e9,
        "unit": "GFLOP/s",
        "cores": oracle.threads(),
        "cores_meaning": "OpenMP threads the oracle ran with, one per logical CPU (hardware thread) this "
                         "process may use",
        "cpu_model": model,
        "logical_cpus_visible": logical,
        "kind": "oracle",
        "sample": "%d rows drawn uniformly at random (seed %d), %d intermediate products, %.1f s" % (
            rows.size, seed, sample_products, dt),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="rmat22", choices=sorted(WORKLOADS) + sorted(PAIR_WORKLOADS))
    ap.add_argument("--panel-products", type=float, default=4e9,
                    help="maximum intermediate products per row panel")
    ap.add_argument("--cpu-products", type=float, default=2.5e9, help="oracle sample size for the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--concurrent", action="store_true", help="run heavy and light work on two streams")
    ap.add_argument("--paper-expansion", action="store_true",
                    help="expand C-hat row by row and split it afterwards (the paper's order)")
    ap.add_argument("--slice-split", action="store_true",
                    help="split at the first level during a slice-order expansion (atomic cursors)")
    ap.add_argument("--level-by-level", action="store_true",
                    help="with two levels, write the first level out and split it in a pass of its own")
    ap.add_argument("--tau", type=int, default=0, help="heavy threshold (0: the planner's)")
    ap.add_argument("--pattern-reuse", action="store_true",
                    help="after the timed steps, also time one values-only re-run per panel (new values of A "
                         "and B on the kept patterns) against the full product on the same plans")
    ap.add_argument("--cache-probe", action="store_true",
                    help="also report the rate of random 128-byte line reads against the working-set size "
                         "(2 MiB .. 4 GiB)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: it measures the single-GPU hot path "
              "(row panels are independent; a multi-GPU run would shard panels, which is not built)",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import workloads
    from paper_2607_22866_amd import gmagnus as g

    g.load()
    if not torch.cuda.is_available():
        raise RuntimeError("no GPU visible")
    torch.cuda.set_device(0)
    pair = args.config in PAIR_WORKLOADS
    cfg = workloads.PAIRS[args.config] if pair else workloads.CONFIGS[args.config]
    t0 = time.perf_counter()
    if pair:
        A, B = cfg.make()
    else:
        A = B = cfg.make()
    log("generated %s: n=%d nnz(A)=%d nnz(B)=%d in %.1fs" % (args.config, A.n_rows, A.nnz, B.nnz,
                                                             time.perf_counter() - t0))
    dA = g.DeviceCSR.from_host(A)
    dB = g.DeviceCSR.from_host(B) if pair else dA
    torch.cuda.synchronize()
    peaks = measured_peaks(g)
    copy_gbs = peaks["copy"]
    log("probe bandwidths (GB/s): " + ", ".join("%s %.0f" % kv for kv in peaks.items()))

    bounds = g.split_panels(dA, dB, int(args.panel_products))
    log("%d row panels (max %.2g products each)" % (len(bounds) - 1, args.panel_products))
    acc_warm = {}
    c_bufs = [None, None]
    extra = ((g.FLAG_CONCURRENT_STREAMS if args.concurrent else 0) | (g.FLAG_PAPER_EXPANSION if args.paper_expansion else 0) |
             (g.FLAG_SLICE_SPLIT if args.slice_split else 0) | (g.FLAG_LEVEL_BY_LEVEL if args.level_by_level else 0))
    for w in range(args.warmup):
        t = time.perf_counter()
        run_step(g, dA, dB, bounds, False, acc_warm, c_bufs, extra, args.tau)
        torch.cuda.synchronize()
        log("warmup %d: %.3fs" % (w, time.perf_counter() - t))

    acc = {}
    products = nnz = 0
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for s in range(args.steps):
        t = time.perf_counter()
        bounds = g.split_panels(dA, dB, int(args.panel_products))
        products, nnz = run_step(g, dA, dB, bounds, True, acc, c_bufs, extra, args.tau)
        torch.cuda.synchronize()
        log("step %d: %.3fs" % (s, time.perf_counter() - t))
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms_per_step = 1000.0 * elapsed / args.steps
    gflops = 2.0 * products / (elapsed / args.steps) / 1e9

    kernels = {}
    for k, rec in acc.items():
        if k.startswith("_"):
            continue
        ms, launches, byts = rec
        if launches == 0 and ms == 0:
            continue
        kernels[k] = {"ms_per_step": ms / args.steps, "launches_per_step": launches / args.steps,
                      "gb_per_step": byts / args.steps / 1e9,
                      "achieved_gbs": (byts / (ms / 1000.0) / 1e9) if ms > 0 else None}
    single = {k: v for k, v in kernels.items() if k in SINGLE_KERNEL_CLASSES and v["launches_per_step"] > 0}
    dom = max(single, key=lambda k: single[k]["ms_per_step"]) if single else None
    roofline = None
    if dom:
        d = kernels[dom]
        kname = SINGLE_KERNEL_CLASSES[dom]
        levels = acc.get("_levels", set())
        if dom == "expand" and (args.paper_expansion or levels == {0}):
            kname = "k_expand"  # also the only expansion without a multisplit level
        elif dom == "expand" and args.slice_split:
            kname = "k_expand_split"
        elif dom == "expand" and (args.level_by_level or levels != {2}):
            kname = "k_expand_rows"
        bpl = d["gb_per_step"] * 1e9 / d["launches_per_step"]
        ms = d["ms_per_step"] / d["launches_per_step"]
        achieved = bpl / (ms / 1000.0) / 1e9
        roofline = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic(kname, args.config),
                    "kernel": kname, "algorithmic_bytes_per_launch": bpl, "avg_launch_ms": ms,
                    "launches_per_step": d["launches_per_step"], "frac_of_copy": achieved / copy_gbs}
    heavy_ms = sum(kernels[k]["ms_per_step"] for k in HEAVY_KERNELS if k in kernels)
    heavy_gb = sum(kernels[k]["gb_per_step"] for k in HEAVY_KERNELS if k in kernels)
    all_ms = sum(v["ms_per_step"] for v in kernels.values())
    all_gb = sum(v["gb_per_step"] for v in kernels.values())

    out = {
        "metric": METRIC.replace("A·A", "A·B") if pair else METRIC,
        "value": gflops,
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": (PAIR_WORKLOADS if pair else WORKLOADS)[args.config], "name": args.config,
                   "seed": cfg.seed, "n": A.n_rows, "nnz_a": A.nnz, "nnz_b": B.nnz, "products": products,
                   "products_heavy": acc.get("_heavy", 0) // max(args.steps, 1), "nnz_c": nnz, "panels": len(bounds) - 1,
                   "panel_products": args.panel_products},
        "achieved_hbm_gbs": {"heavy_path_kernels": heavy_gb / (heavy_ms / 1000.0) if heavy_ms else None,
                             "heavy_path_frac": (heavy_gb / (heavy_ms / 1000.0)) / HBM_PEAK_GBS if heavy_ms else None,
                             "heavy_path_frac_of_copy": (heavy_gb / (heavy_ms / 1000.0)) / copy_gbs
                             if heavy_ms else None,
                             "copy_peak": copy_gbs,
                             "probe_peaks": peaks,
                             "all_kernels": all_gb / (all_ms / 1000.0) if all_ms else None,
                             "end_to_end": all_gb / (elapsed / args.steps)},
        "roofline": roofline,
        "kernels": kernels,
        "kernel_ms_sum_per_step": all_ms,
        "check_flags": 0,
    }
    if args.pattern_reuse:
        t_full, t_vals = reuse_pass(g, dA, dB, bounds, c_bufs, extra, args.tau)
        out["pattern_reuse"] = {"full_ms": 1000.0 * t_full, "values_only_ms": 1000.0 * t_vals,
                                "values_only_gflops": 2.0 * products / t_vals / 1e9,
                                "speedup": t_full / t_vals,
                                "note": "panel by panel, synchronised around each phase; full = plan + symbolic + "
                                        "numeric with the pattern kept, values only = gmagnus_update_values + numeric"}
    if args.cache_probe:
        out["cache_probe_gbs"] = cache_probe(g)
    if not args.no_cpu_baseline:
        ip = g.row_products(dA, dB).cpu().numpy()
        log("timing the oracle on a sample of about %.2g products" % args.cpu_products)
        out["cpu_baseline"] = cpu_baseline(A, B, ip, args.cpu_products)
        del np
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
