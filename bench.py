"""Throughput of the kNN-OD / LOF hot path on one MI355X.

With no --workload, the headline line is the largest configuration, C5
(n = 4,000,000, d = 8, k = 5, kNN-OD), and the line carries C1-C4 as
sub-results under "configs", each run as its workload specifies it (filter
precision; LOF where the workload asks for it).

One step = one library call on the whole workload: prep, fused distance tiles
with top-K' selection, certificate + exact recheck, fallback and the scores
of every point.  The detector is the workload's own (tod_lof for C1 and C2,
tod_knn_score for C3-C5) unless --detector says otherwise (knn, lof, abod,
cof).  Inputs are resident in HBM before timing starts.
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
    ap.add_argument("--workload", default=None,
                    help="one workload only (C1-C5, N1, L1); default: C5 as the headline with "
                         "C1-C4 as sub-results")
    ap.add_argument("--precision", default=None,
                    help="filter precision (auto, fp32, fp16, bf16); default: the workload's")
    ap.add_argument("--detector", default=None, choices=("lof", "knn", "abod", "cof"),
                    help="what one step computes on a kNN workload; default: the workload's "
                         "(LOF with the kNN score for C1 and C2, the kNN score for C3-C5)")
    ap.add_argument("--score", default="kth", choices=("kth", "mean", "median", "sum"),
                    help="kNN score of the step")
    ap.add_argument("--sub-steps", type=int, default=5,
                    help="timed steps of each sub-result (one warm-up step each)")
    ap.add_argument("--no-sub", action="store_true", help="headline line without sub-results")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target wall time of the oracle baseline sample (N1, L1)")
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


def cpu_baseline(x, k, rows, lof_full=False):
    """The oracle (exact fp64 brute force, every host core in the affinity
    mask) on the seeded sample `rows` of query rows, each scanned against the
    whole reference set.  With lof_full the whole workload is run instead:
    the oracle's kNN of every row and its LOF."""
    from oracle import oracle
    n = x.shape[0]
    t0 = time.perf_counter()
    if lof_full:
        oidx, odist = oracle.knn_self(x, k)
        oracle.lof(oidx, odist)
        m = n
    else:
        oracle.knn_self(x, k, rows=rows)
        m = len(rows)
    t = time.perf_counter() - t0
    what = ("exact fp64 kNN (k=%d) and LOF of all %d rows" % (k, n) if lof_full else
            "exact fp64 kNN (k=%d) of %d seeded query rows (default_rng sample of the workload) "
            "against all %d reference rows" % (k, m, n))
    return {
        "value": m / t,
        "unit": "points/s",
        "cores": oracle.default_threads(),
        "kind": "oracle",
        "sample": "%s, %.2f s of oracle time (%.3g pairs/s)" % (what, t, float(m) * n / t),
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
    opts = tod.options(precision=args.precision or w.precision, exclude_self=True)
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
    opts = tod.options(precision=args.precision or w.precision)
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




# Peak VALU issue rate: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz = 3.93e13 lane
# operations per second (fp32, unpacked, one operation per lane per clock).
PEAK_VALU_OPS = 39.32        # T lane-ops/s


def tile_rooflines(prec, d, pairs, launches, tile_ms):
    """Both views of the dominant kernel, the fused distance tile, per launch.

    mfma: the cross-term's 2d flop per pair (d as given, not padded) against
    the dense MFMA peak (an fp32 filter: against the fp32 vector peak).
    alu:  the selection's one fp32 compare per pair (an fp32 filter adds its
    d multiply-adds) against the VALU issue peak.
    The binding view is the one whose floor time is longer."""
    launch_s = tile_ms / launches * 1e-3
    per_launch = pairs / launches
    if prec == "fp32":
        mf_peak, ops_pair = PEAK_VALU_F32, d + 1.0
    else:
        mf_peak, ops_pair = PEAK_MFMA_F16, 1.0
    mf = 2.0 * d * per_launch / launch_s / 1e12
    alu = ops_pair * per_launch / launch_s / 1e12
    views = {
        "mfma": {"bound": "mfma", "achieved": round(mf, 3), "peak": mf_peak, "unit": "TFLOP/s",
                 "frac": round(mf / mf_peak, 4),
                 "ops": "2d flop per pair (cross-term)"},
        "alu": {"bound": "alu", "achieved": round(alu, 3), "peak": PEAK_VALU_OPS,
                "unit": "TFLOP/s", "frac": round(alu / PEAK_VALU_OPS, 4),
                "ops": "%g fp32 VALU op per pair (%s)" % (
                    ops_pair, "threshold compare" if prec != "fp32" else "FMA chain + compare")},
    }
    floor_mf = 2.0 * d * pairs / (mf_peak * 1e12)
    floor_alu = ops_pair * pairs / (PEAK_VALU_OPS * 1e12)
    bind = "mfma" if floor_mf >= floor_alu else "alu"
    return bind, views


def bench_knn(w, x_host, steps, warmup, precision, detector, score="kth"):
    """Time `steps` calls of the workload's detector; returns the measurement."""
    import numpy as np
    import torch

    from paper_2110_14007_amd import tod

    n, d, k = x_host.shape[0], x_host.shape[1], w.k
    dev = torch.device("cuda:0")
    x = torch.from_numpy(x_host).to(dev)
    opts = tod.options(precision=precision, query_block=w.query_block, score=score)
    ws = tod.Workspace()
    out = (torch.empty(n, dtype=torch.float32, device=dev),
           torch.empty(n, dtype=torch.float32, device=dev))

    def step(st=None):
        if detector == "lof":
            tod.tod_lof(x, k, opts, workspace=ws, out=out, stats=st)
        elif detector == "knn":
            tod.tod_knn_score(x, k, opts, workspace=ws, stats=st)
        elif detector == "cof":
            tod.tod_cof(x, min(k, 63), opts, workspace=ws, stats=st)
        else:
            tod.tod_abod(x, min(k, 64), opts, workspace=ws, stats=st)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    stats = []
    t0 = time.perf_counter()
    for _ in range(steps):
        st = tod.new_stats()
        step(st)
        stats.append(st.as_dict())
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / steps
    del x, ws, out
    torch.cuda.empty_cache()

    def avg(key):
        return float(np.mean([s[key] for s in stats]))

    prec = stats[0]["precision"]
    launches = stats[0]["tile_launches"]
    pairs = float(n) * float(n)
    bind, views = tile_rooflines(prec, d, pairs, launches, avg("ms_tile"))
    recheck = recheck_roofline(n, d, k, stats[0]["kprime"], stats[0]["ref_splits"],
                               avg("ms_recheck"))
    return {
        "n": n, "d": d, "k": k, "detector": detector, "score": score, "prec": prec,
        "ms_step": ms_step, "value": n / (ms_step * 1e-3), "pairs_s": pairs / (ms_step * 1e-3),
        "phase_ms": {key: round(avg(key), 4) for key in
                     ("ms_prep", "ms_tile", "ms_recheck", "ms_fallback", "ms_score", "ms_total")},
        "kprime": stats[0]["kprime"], "ref_splits": stats[0]["ref_splits"],
        "query_block": stats[0]["query_block"], "blocks": stats[0]["blocks"],
        "launches": launches, "launch_ms": avg("ms_tile") / launches,
        "rows_fallback": stats[0]["rows_fallback"], "bind": bind, "views": views,
        "recheck": recheck,
    }


def recheck_roofline(n, d, k, kprime, splits, ms):
    """The recheck against the HBM peak on its algorithmic bytes per row: the
    S lists (8 B per entry), the measured candidates' fp32 rows and the query's
    own, its squared norm and radius, and k neighbours written (index and
    distance, 12 B each) plus the k-th distance.  Lists of up to 32 entries
    over rows of up to 64 elements (a multiple of 4) measure all K'
    candidates; otherwise the first pass measures k + 8."""
    lanes = kprime <= 32 and d <= 64 and d % 4 == 0
    measured = kprime if lanes else min(k + 8, kprime)
    per_row = splits * kprime * 8 + (measured + 1) * 4 * d + 16 + k * 12 + 8
    gbs = n * per_row / (ms * 1e-3) / 1e9 if ms > 0 else 0.0
    return {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(gbs / PEAK_HBM_GBS, 4), "bytes_per_row": per_row,
            "kernel": ("recheck_lanes<K'=%d>" if lanes else "recheck<K'=%d>") % kprime,
            "ms": round(ms, 4)}


def knn_roofline(wname, m):
    """The line's `roofline` object: the binding view of the tile kernel, the
    other view beside it, and the recorded HBM traffic per launch."""
    kname = "tile<%s,K'=%d>" % (m["prec"], m["kprime"])
    r = dict(m["views"][m["bind"]])
    r["traffic"] = recorded_traffic(wname, kname)
    r["kernel"] = kname
    r["launch_ms"] = round(m["launch_ms"], 4)
    other = "alu" if m["bind"] == "mfma" else "mfma"
    r["other_view"] = m["views"][other]
    return r


def knn_defaults(w, args):
    precision = args.precision or w.precision
    detector = args.detector or ("lof" if w.lof else "knn")
    return precision, detector


def knn_line(args, w):
    """The JSON line of one kNN workload (headline fields)."""
    from paper_2110_14007_amd import workloads
    x_host, _ = workloads.generate(w.name)
    precision, detector = knn_defaults(w, args)
    m = bench_knn(w, x_host, args.steps, args.warmup, precision, detector, args.score)
    line = {
        "metric": METRIC,
        "value": round(m["value"], 1),
        "unit": "points/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(m["ms_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32+f64" if m["prec"] == "fp32" else "%s+f64" % m["prec"].replace("fp", "f"),
        "data": "synthetic",
        "config": {"workload": "%s: %s" % (w.name, w.description), "n": m["n"], "d": m["d"],
                   "k": m["k"], "detector": detector, "score": args.score,
                   "filter_precision": m["prec"], "kprime": m["kprime"],
                   "ref_splits": m["ref_splits"], "query_block": m["query_block"],
                   "parallelism": "single GPU"},
        "pairs_per_s": m["pairs_s"],
        "phase_ms": m["phase_ms"],
        "rows_fallback": m["rows_fallback"],
        "roofline": knn_roofline(w.name, m),
        "recheck_roofline": m["recheck"],
    }
    return line, x_host


def sub_result(args, w, precision=None, label=None):
    """One configuration as a sub-result: its own precision and detector,
    ms/step, tile time, both roofline views and the oracle's rate on a seeded
    sample of its rows (C1: the whole oracle, kNN and LOF)."""
    from paper_2110_14007_amd import workloads
    x_host, _ = workloads.generate(w.name)
    prec_w, detector = knn_defaults(w, args)
    precision = precision or prec_w
    m = bench_knn(w, x_host, args.sub_steps, 1, precision, detector)
    r = {"workload": label or w.name, "n": m["n"], "d": m["d"], "k": m["k"],
         "detector": detector, "filter_precision": m["prec"], "kprime": m["kprime"],
         "ms_per_step": round(m["ms_step"], 4), "points_per_s": round(m["value"], 1),
         "pairs_per_s": m["pairs_s"], "tile_ms": round(m["phase_ms"]["ms_tile"], 4),
         "phase_ms": m["phase_ms"], "rows_fallback": m["rows_fallback"],
         "roofline": knn_roofline(w.name, m), "recheck_roofline": m["recheck"],
         "steps": args.sub_steps}
    if not args.no_cpu_baseline:
        if w.name == "C1":
            r["oracle"] = cpu_baseline(x_host, w.k, None, lof_full=True)
        else:
            r["oracle"] = cpu_baseline(x_host, w.k, workloads.sample_rows(w.name, count=256))
    return r


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: --gpus %d is not supported (the path runs on "
              "one GPU; no multi-GPU mode is built)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    if args.copy_mib:
        copy_calibration(args.copy_mib, args.steps)
        return
    from paper_2110_14007_amd import workloads

    name = args.workload or "C5"
    w = workloads.WORKLOADS[name]
    if w.name.startswith("N"):
        bench_nwr(args, w)
        return
    if w.name.startswith("L"):
        bench_loci(args, w)
        return
    line, x_host = knn_line(args, w)
    if not args.no_cpu_baseline:
        if w.name == "C1":
            line["cpu_baseline"] = cpu_baseline(x_host, w.k, None, lof_full=True)
        else:
            line["cpu_baseline"] = cpu_baseline(x_host, w.k, workloads.sample_rows(w.name))
    del x_host
    if args.workload is None and not args.no_sub:
        subs = []
        for sub in ("C1", "C2", "C3", "C4"):
            subs.append(sub_result(args, workloads.WORKLOADS[sub]))
            print("# %s done" % sub, file=sys.stderr, flush=True)
        # the library's default filter at C4 (fp16) beside the workload's bf16
        subs.append(sub_result(args, workloads.WORKLOADS["C4"], precision="auto",
                               label="C4 (library default filter)"))
        line["configs"] = subs
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
