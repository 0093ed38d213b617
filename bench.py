"""Throughput of the kNN-OD / LOF hot path on one MI355X.

One step = one tod_lof call on the whole workload: prep, fused distance tiles
with top-K' selection, certificate + exact recheck, fallback, kNN-OD score
and LOF for every point (--detector knn: the kNN score alone; --detector abod
or cof: ABOD or COF from the same lists).  Inputs are resident in HBM before timing starts.
For a neighbours-within-range workload (--workload N1) one step is one
tod_nwr call as the paper defines the operator (the indices of the pairs in
range): prep, the range tile's count and fill passes, exact verification of
the uncertain pairs and the CSR output.  For the LOCI workload (--workload L1)
one step is one tod_loci call: neighbours within the largest radius, then the
per-radius neighbourhood counts, sums, MDEF, score and flag of every point.

Prints ONE JSON line (see the design doc for the field definitions).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "kNN-OD scored points/sec and distance-pairs/sec (1 MI355X); % of MFMA/HBM roofline"
# Peaks used for the roofline fraction (MI355X: 256 CUs x 4 SIMD, 2.4 GHz).
PEAK_MFMA_F16 = 2500.0      # TFLOP/s, dense fp16 / bf16 MFMA
PEAK_VALU_F32 = 157.3       # TFLOP/s, published fp32 vector peak (packed FMA)
PEAK_HBM_GBS = 8000.0       # GB/s, HBM3E


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="C2")
    ap.add_argument("--precision", default="auto")
    ap.add_argument("--detector", default="lof", choices=("lof", "knn", "abod", "cof"),
                    help="what one step computes on a kNN workload: LOF (with the kNN score, "
                         "the default), the kNN score alone, ABOD or COF")
    ap.add_argument("--score", default="kth", choices=("kth", "mean", "median", "sum"),
                    help="kNN score of the step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target wall time of the oracle baseline sample")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="instead of the benchmark, run a plain device-to-device copy of this "
                         "many MiB (calibrates the HBM byte counters against a known size)")
    return ap.parse_args()


def copy_calibration(mib, steps):
    """A plain copy kernel of known size: reads and writes mib MiB per launch."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.arange(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    print(json.dumps({"copy_mib": mib, "bytes_read": n * 4, "bytes_written": n * 4,
                      "ms_per_copy": round(ms, 4),
                      "GB_s": round(2 * n * 4 / (ms * 1e-3) / 1e9, 1)}), flush=True)


def cpu_baseline(x, k, target_s):
    """The oracle (exact fp64 brute force) on a bounded sample of query rows.

    Rows are taken in a seeded random order without repetition, in batches
    that double until about target_s seconds of oracle time have been spent.
    """
    import numpy as np

    from oracle import oracle
    n = x.shape[0]
    order = np.random.default_rng(2024).permutation(n).astype(np.int64)
    rows_done, t_total = 0, 0.0
    batch = 256
    while t_total < target_s and rows_done < n:
        m = min(batch, n - rows_done)
        rows = np.sort(order[rows_done:rows_done + m])
        t0 = time.perf_counter()
        oracle.knn_self(x, k, rows=rows)
        t_total += time.perf_counter() - t0
        rows_done += m
        if t_total < target_s / 4:
            batch *= 2
    return {
        "value": rows_done / t_total,
        "unit": "points/s",
        "cores": oracle.default_threads(),
        "kind": "oracle",
        "sample": "exact fp64 kNN (k=%d) of %d distinct seeded-random query rows against all %d "
                  "reference rows, %.1f s of oracle time; the O(n k) LOF tail is not timed"
                  % (k, rows_done, n, t_total),
    }


# Sources that decide what the tile kernels execute: the kernels themselves,
# their shared headers and the planner that picks their template arguments.
TILE_SOURCES = ("api.hip", "tod_internal.h", "wave.h", "halfwave.h", "tile.h", "tile_f32.hip",
                "tile_f16.hip", "tile_bf16.hip", "mtile.h", "mtile_f16.hip", "mtile_bf16.hip",
                "order.hip", "rtile.h", "rtile_f16.hip", "rtile_bf16.hip", "nwr.hip", "loci.hip")


def kernel_sources_digest():
    """sha256 over the tile kernels' sources; a counter record applies only to this digest."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2110_14007_amd", "csrc")
    h = hashlib.sha256()
    for name in TILE_SOURCES:
        h.update(name.encode())
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(f.read())
    with open(os.path.join(ROOT, "include", "tod.h"), "rb") as f:
        h.update(f.read())
    return h.hexdigest()


def recorded_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary, or
    None when the summary is missing or was taken on different kernel sources."""
    path = os.path.join(ROOT, "profiles", "hbm_counters_%s.txt" % workload)
    if not os.path.exists(path):
        return None
    digest, traffic = None, None
    with open(path) as f:
        for line in f:
            if line.startswith("csrc_sha256:"):
                digest = line.split()[1]
            elif line.startswith("traffic_bytes_per_launch:") and kernel in line:
                traffic = float(line.split()[1])
    if digest != kernel_sources_digest():
        return None
    return traffic


def cpu_baseline_nwr(x, phi, target_s):
    """The oracle's neighbours within range on a bounded sample of query rows."""
    import numpy as np

    from oracle import oracle
    n = x.shape[0]
    order = np.random.default_rng(2024).permutation(n).astype(np.int64)
    rows_done, t_total, batch = 0, 0.0, 64
    while t_total < target_s and rows_done < n:
        m = min(batch, n - rows_done)
        rows = np.sort(order[rows_done:rows_done + m])
        t0 = time.perf_counter()
        oracle.nwr(x, x, phi, exclude_self=True, rows=rows)
        t_total += time.perf_counter() - t0
        rows_done += m
        if t_total < target_s / 4:
            batch *= 2
    return {
        "value": rows_done / t_total,
        "unit": "points/s",
        "cores": oracle.default_threads(),
        "kind": "oracle",
        "sample": "exact fp64 neighbours within range (phi=%g) of %d distinct seeded-random "
                  "query rows against all %d reference rows, %.1f s of oracle time"
                  % (phi, rows_done, n, t_total),
    }


def bench_nwr(args, w):
    """One step = one tod_nwr call (X against itself, self excluded, indices only)."""
    import numpy as np
    import torch

    from paper_2110_14007_amd import tod, workloads

    x_host, _ = workloads.generate(w.name)
    n, d = x_host.shape
    phi = float(w.extra["phi"])
    x = torch.from_numpy(x_host).to("cuda:0")
    opts = tod.options(precision=args.precision, exclude_self=True)
    ws = tod.Workspace()
    rp, idx, _ = tod.tod_nwr(x, x, phi, opts, workspace=ws, with_dist=False)  # sizes the outputs
    cap = int(idx.numel())
    for _ in range(max(args.warmup - 1, 0)):
        tod.tod_nwr(x, x, phi, opts, workspace=ws, capacity=cap, with_dist=False)
    torch.cuda.synchronize()
    stats = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        st = tod.new_stats()
        tod.tod_nwr(x, x, phi, opts, workspace=ws, capacity=cap, stats=st, with_dist=False)
        stats.append(st.as_dict())
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps

    def avg(key):
        return float(np.mean([s[key] for s in stats]))

    prec = stats[0]["precision"]
    launches = stats[0]["tile_launches"]
    # the count pass and the fill passes each evaluate every pair once
    flops = 2.0 * 2.0 * d * float(n) * float(n)
    tile_ms = avg("ms_tile") / launches
    achieved = flops / launches / (tile_ms * 1e-3) / 1e12
    kname = "range_tile<%s,d=%d>" % (prec, d)
    line = {
        "metric": METRIC,
        "value": round(n / (ms_step * 1e-3), 1),
        "unit": "points/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "%s+f64" % prec.replace("fp", "f"),
        "data": "synthetic",
        "config": {"workload": "%s: %s" % (w.name, w.description), "n": n, "d": d, "phi": phi,
                   "filter_precision": prec, "ref_splits": stats[0]["ref_splits"],
                   "batches": stats[0]["blocks"], "parallelism": "single GPU"},
        "pairs_per_s": float(n) * float(n) / (ms_step * 1e-3),
        "pairs_in_range": stats[0]["pairs_in_range"],
        "pairs_candidate": stats[0]["pairs_candidate"],
        "pairs_uncertain": stats[0]["pairs_uncertain"],
        "phase_ms": {key: round(avg(key), 4) for key in ("ms_prep", "ms_tile", "ms_recheck",
                                                         "ms_total")},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_MFMA_F16,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_MFMA_F16, 4),
                     "traffic": recorded_traffic(w.name, kname), "kernel": kname,
                     "launch_ms": round(tile_ms, 4)},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_nwr(x_host, phi, args.cpu_seconds)
    print(json.dumps(line), flush=True)


def cpu_baseline_loci(x, p, target_s):
    """The oracle's LOCI on a bounded sample: the first m rows of the workload
    taken as a point set of their own (LOCI of n points costs O(n^2) pairs,
    so the oracle's pair rate divided by the workload's n is its point rate
    on the whole workload)."""
    from oracle import oracle
    n = x.shape[0]
    m, t = 2000, 0.0
    while True:
        t0 = time.perf_counter()
        oracle.loci(x[:m], p["radii"], p["alpha"], p["n_min"], p["k_sigma"])
        t = time.perf_counter() - t0
        if t >= target_s / 4 or m >= min(n, 12000):
            break
        m = min(2 * m, n, 12000)
    pairs_s = float(m) * float(m) / t
    return {
        "value": pairs_s / n,
        "unit": "points/s",
        "cores": 1,
        "kind": "oracle",
        "sample": "numpy fp64 LOCI of the first %d rows as their own point set (%.3g pairs in "
                  "%.1f s = %.3g pairs/s), divided by n = %d pairs per point"
                  % (m, float(m) * m, t, pairs_s, n),
    }


def bench_loci(args, w):
    """One step = one tod_loci call: neighbours within the largest radius
    (prep, range tile count and fill passes, exact verification, CSR), then
    the LOCI count and sum kernels."""
    import numpy as np
    import torch

    from paper_2110_14007_amd import tod, workloads

    x_host, _ = workloads.generate(w.name)
    n, d = x_host.shape
    p = w.extra
    x = torch.from_numpy(x_host).to("cuda:0")
    opts = tod.options(precision=args.precision)
    ws = tod.Workspace()
    st = tod.new_stats()
    tod.tod_loci(x, p["radii"], p["alpha"], p["n_min"], p["k_sigma"], opts, workspace=ws,
                 stats=st)  # sizes the workspace
    cap = int(st.pairs_in_range)

    def step(s=None):
        return tod.tod_loci(x, p["radii"], p["alpha"], p["n_min"], p["k_sigma"], opts,
                            capacity=cap, grow=False, workspace=ws, stats=s)

    for _ in range(max(args.warmup - 1, 0)):
        step()
    torch.cuda.synchronize()
    stats = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        s = tod.new_stats()
        step(s)
        stats.append(s.as_dict())
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps

    def avg(key):
        return float(np.mean([s[key] for s in stats]))

    prec = stats[0]["precision"]
    nl = len(p["radii"])
    nls = 8 if nl <= 8 else (16 if nl <= 16 else 32)
    pairs = float(stats[0]["pairs_in_range"])
    # Algorithmic HBM bytes of the two LOCI kernels: each reads the pair ids
    # (8 B) and the radius index (1 B, written by the first); the count tables
    # (2 x n x nls int32) are written once and read once.  The rows and the
    # count rows gathered per pair are cache-resident (x: 16 n B, table: 4 n nls B).
    loci_bytes = pairs * (8 + 1) * 2 + pairs * 1 + 2.0 * n * nls * 4 * 2
    loci_ms = avg("ms_score")
    achieved = loci_bytes / (loci_ms * 1e-3) / 1e9
    line = {
        "metric": METRIC,
        "value": round(n / (ms_step * 1e-3), 1),
        "unit": "points/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "%s+f64" % prec.replace("fp", "f"),
        "data": "synthetic",
        "config": {"workload": "%s: %s" % (w.name, w.description), "n": n, "d": d,
                   "radii": [round(r, 6) for r in p["radii"]], "alpha": p["alpha"],
                   "n_min": p["n_min"], "k_sigma": p["k_sigma"], "filter_precision": prec,
                   "parallelism": "single GPU"},
        "pairs_per_s": float(n) * float(n) / (ms_step * 1e-3),
        "pairs_in_range": int(pairs),
        "phase_ms": {key: round(avg(key), 4) for key in ("ms_prep", "ms_tile", "ms_recheck",
                                                         "ms_score", "ms_total")},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                     "traffic": recorded_traffic(w.name, "loci_count+loci_sum"),
                     "kernel": "loci_count+loci_sum", "launch_ms": round(loci_ms, 4)},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline_loci(x_host, p, args.cpu_seconds)
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: --gpus %d is not supported (the path has no "
              "multi-GPU mode)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    if args.copy_mib:
        copy_calibration(args.copy_mib, args.steps)
        return
    import numpy as np
    import torch

    from paper_2110_14007_amd import tod, workloads

    w = workloads.WORKLOADS[args.workload]
    if w.name.startswith("N"):
        bench_nwr(args, w)
        return
    if w.name.startswith("L"):
        bench_loci(args, w)
        return
    x_host, _ = workloads.generate(args.workload)
    n, d, k = x_host.shape[0], x_host.shape[1], w.k
    dev = torch.device("cuda:0")
    x = torch.from_numpy(x_host).to(dev)
    opts = tod.options(precision=args.precision, query_block=w.query_block, score=args.score)
    ws = tod.Workspace()
    out = (torch.empty(n, dtype=torch.float32, device=dev),
           torch.empty(n, dtype=torch.float32, device=dev))

    def step(st=None):
        if args.detector == "lof":
            tod.tod_lof(x, k, opts, workspace=ws, out=out, stats=st)
        elif args.detector == "knn":
            tod.tod_knn_score(x, k, opts, workspace=ws, stats=st)
        elif args.detector == "cof":
            tod.tod_cof(x, min(k, 63), opts, workspace=ws, stats=st)
        else:
            tod.tod_abod(x, min(k, 64), opts, workspace=ws, stats=st)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stats = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        st = tod.new_stats()
        step(st)
        stats.append(st.as_dict())
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    value = n / (ms_step * 1e-3)
    pairs_s = float(n) * float(n) / (ms_step * 1e-3)

    def avg(key):
        return float(np.mean([s[key] for s in stats]))

    prec = stats[0]["precision"]
    launches = stats[0]["tile_launches"]
    tile_ms = avg("ms_tile") / launches  # average duration of one tile launch
    flops_per_launch = 2.0 * d * float(n) * float(n) / launches
    achieved = flops_per_launch / (tile_ms * 1e-3) / 1e12
    if prec == "fp32":
        bound, peak = "alu", PEAK_VALU_F32
    else:
        bound, peak = "mfma", PEAK_MFMA_F16
    kname = "tile<%s,K'=%d>" % (prec, stats[0]["kprime"])
    roofline = {"bound": bound, "achieved": round(achieved, 3), "peak": peak,
                "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                "traffic": recorded_traffic(args.workload, kname),
                "kernel": kname, "launch_ms": round(tile_ms, 4)}
    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "points/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32+f64" if prec == "fp32" else "%s+f64" % prec.replace("fp", "f"),
        "data": "synthetic",
        "config": {"workload": "%s: %s" % (w.name, w.description), "n": n, "d": d, "k": k,
                   "detector": args.detector, "score": args.score,
                   "filter_precision": prec, "kprime": stats[0]["kprime"],
                   "ref_splits": stats[0]["ref_splits"], "query_block": stats[0]["query_block"],
                   "parallelism": "single GPU"},
        "pairs_per_s": pairs_s,
        "phase_ms": {key: round(avg(key), 4) for key in
                     ("ms_prep", "ms_tile", "ms_recheck", "ms_fallback", "ms_score", "ms_total")},
        "rows_fallback": stats[0]["rows_fallback"],
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(x_host, k, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
