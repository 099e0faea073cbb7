#!/usr/bin/env python3
"""Benchmark of the MTI k-means hot path on one MI355X.

A step is one Lloyd iteration with MTI pruning: centroid table and drift,
bound update and Clause-1 test, fused distance + argmin of the survivors,
per-cluster reduction into new centroids and the convergence counters.  The
timed region enqueues K consecutive iterations of a run started from the
workload's seeded initial centroids (inputs already resident in HBM) and is
bracketed by device synchronisation; the reported value is iterations per
second.  Per-kernel device times come from HIP events recorded by the
library on its stream around every launch.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--spherical] [--no-cpu-baseline]
    python bench.py --kmeanspp [--workload NAME]      (k-means++ seeding)
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
MFMA_F32_PEAK_TFS = 157.3   # MI355X dense float32 matrix peak
DEFAULT_WORKLOAD = "aniso-8M-d16-k10"
METRIC = "k-means iters/sec + effective dist evals/sec; % HBM peak (low d) / % MFMA (big k·d)"


def log(msg: str) -> None:
    print("[bench] " + msg, file=sys.stderr, flush=True)


# Dominant (assignment-step) kernel of each library path.
DOMINANT_KERNEL = {"stream-d16": "k_inc", "stream-d16-full": "k_small", "lds-vector": "k_assign",
                   "lds-mfma": "k_assign", "lds-elkan": "k_assign",
                   "global-mfma": "k_mfma_large"}
# Sources of each dominant kernel: the hardware byte counts of a committed
# profile summary are used only while these files are unchanged.
KERNEL_SOURCES = {
    "k_small": ["km_small.hip", "km_device.h", "km_internal.h"],
    "k_inc": ["km_small.hip", "km_device.h", "km_internal.h"],
    "k_assign": ["km_kernels.hip", "km_device.h", "km_internal.h"],
    "k_mfma_large": ["km_large.hip", "km_device.h", "km_internal.h"],
    "k_pp_step": ["km_pp.hip", "km_device.h", "km_internal.h"],
}


def _code_only(text: str) -> str:
    """Source text without comments and with whitespace collapsed, so that the
    hash follows the code (string literals hold no comment markers here)."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES.get(kernel, []):
        with open(os.path.join(ROOT, "paper_1902_09527_amd", "csrc", f), encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the rocprofv3 FETCH_SIZE / WRITE_SIZE summary in
    profiles/<kernel>_<workload>.txt, scaled by the plain-copy calibration
    recorded there; None when there is no summary or the kernel changed."""
    path = os.path.join(ROOT, "profiles", "%s_%s.txt" % (kernel, workload))
    if not os.path.exists(path):
        return None, "no profile summary"
    vals = {}
    for line in open(path):
        if "=" in line and line.strip().startswith("pmc."):
            key, val = line.split("=", 1)
            vals[key.strip()] = val.strip()
    try:
        if vals["pmc.kernel_source_sha256"] != kernel_source_hash(kernel):
            return None, "kernel changed since the counters were taken"
        fetch = float(vals["pmc.FETCH_SIZE_KiB_per_dispatch"]) * float(vals["pmc.FETCH_SIZE_scale"])
        write = float(vals["pmc.WRITE_SIZE_KiB_per_dispatch"]) * float(vals["pmc.WRITE_SIZE_scale"])
    except (KeyError, ValueError):
        return None, "incomplete profile summary"
    return (fetch + write) * 1024.0, os.path.relpath(path, ROOT)


def roofline_entry(kernel: str, workload: str, bytes_per_launch: float, launch_ms: float, what: str) -> dict:
    """HBM roofline of one kernel: algorithmic bytes per launch over its mean
    launch time (HIP events), against the 8 TB/s peak."""
    achieved = bytes_per_launch / (launch_ms / 1e3) / 1e9
    traffic, source = measured_traffic(kernel, workload)
    return {"kernel": kernel, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, "traffic": traffic, "traffic_source": source,
            "bytes_per_launch": bytes_per_launch, "bytes_def": what, "kernel_us": launch_ms * 1e3}


def mfma_roofline_entry(kernel: str, workload: str, flops_per_launch: float, launch_ms: float,
                        what: str) -> dict:
    """Matrix-core roofline of one kernel: algorithmic float32 flops per launch
    over its mean launch time (HIP events), against the dense float32 peak."""
    achieved = flops_per_launch / (launch_ms / 1e3) / 1e12
    traffic, source = measured_traffic(kernel, workload)
    return {"kernel": kernel, "bound": "mfma", "achieved": achieved, "peak": MFMA_F32_PEAK_TFS,
            "unit": "TFLOP/s", "frac": achieved / MFMA_F32_PEAK_TFS, "traffic": traffic,
            "traffic_source": source, "flops_per_launch": flops_per_launch, "flops_def": what,
            "kernel_us": launch_ms * 1e3}


def cpu_baseline(X, C0, w, budget_s: float = 15.0, spherical: bool = False) -> dict:
    """Time the CPU oracle (plain float64 Lloyd's or spherical k-means, as it
    stands) on this host."""
    import oracle
    fn = oracle.spherical if spherical else oracle.lloyd
    t0 = time.perf_counter()
    fn(X, C0, 1, 0.0)
    t1 = time.perf_counter() - t0
    iters = int(max(1, min(w.max_iters, budget_s // max(t1, 1e-3))))
    t0 = time.perf_counter()
    r = fn(X, C0, iters, 0.0)
    el = time.perf_counter() - t0
    ips = r["iters"] / el
    return {
        # the spherical oracle is a single-threaded loop
        "value": ips, "unit": "iters/s", "cores": 1 if spherical else oracle.get_threads(), "kind": "oracle",
        "sample": "all %d rows of %s, first %d iterations from the seeded centroids (tol ignored); "
                  "%.3g effective dist evals/s" % (w.n, w.name, r["iters"], ips * w.n * w.k),
    }


def bench_kmeanspp(args, w, X) -> dict:
    """k-means++ seeding of the workload's k seeds: a step is one whole
    seeding (k passes over the points and k - 1 draws)."""
    import numpy as np
    import torch

    import paper_1902_09527_amd as km

    n, d, k = w.n, w.d, w.k
    K = args.steps or 5
    Xg = torch.from_numpy(X).to("cuda:0")
    ws = torch.empty(km.kmeanspp_workspace_bytes(n, d, k) + 256, dtype=torch.uint8, device="cuda:0")
    U = np.random.default_rng(20190225).random((args.warmup + K + 1, k))
    for r in range(args.warmup):
        km.kmeanspp(Xg, k, U[r], workspace=ws)
    torch.cuda.synchronize()
    log("warmup done (%d seedings)" % args.warmup)
    t0 = time.perf_counter()
    for r in range(K):
        km.kmeanspp(Xg, k, U[args.warmup + r], workspace=ws)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    log("timed %d seedings in %.3f ms" % (K, elapsed * 1e3))
    tm = km.kmeanspp(Xg, k, U[-1], workspace=ws, timing=True)["stats"]
    G = (n + 2047) // 2048
    roof = {"kernel": "k_pp_step", "bound": "hbm", "achieved": None, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": None, "traffic": None}
    if k > 1 and tm["later_pass_ms"] > 0:
        # Passes 2..k: D2 and the nearest-seed index of every row read (12 B),
        # the block weight sum written (8 B per 2048 rows), a surviving row
        # read (4d B) and an improved row's D2 and index written (12 B).
        bytes_later = (k - 1) * (12.0 * n + 8.0 * G) + 4.0 * d * (tm["computed"] - n) + 12.0 * tm["improved"]
        roof = roofline_entry("k_pp_step", w.name + "-kmeanspp", bytes_later / (k - 1),
                              tm["later_pass_ms"] / (k - 1),
                              "passes 2..k: 12n (D2, nearest seed) + 8 per block sum + 4d per survivor row "
                              "+ 12 per improved row")
    result = {
        "metric": "k-means++ seedings/s (k seeds each)",
        "value": K / elapsed,
        "unit": "seedings/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": w.name, "method": "kmeans++ seeding", "n": n, "d": d, "k": k,
                   "timed": "%d seedings with seeded uniforms" % K},
        "seeds_per_s": k * K / elapsed,
        "dist_computed_frac": tm["computed"] / float(n * k),
        "kernel_ms_per_step": {"passes": tm["pass_ms"], "draws": tm["draw_ms"]},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        import oracle
        log("cpu baseline (oracle) ...")
        t0 = time.perf_counter()
        oracle.kmeanspp(X, 1, U[-1][:1])
        t1 = time.perf_counter() - t0
        kk = int(max(1, min(k, 15.0 // max(t1, 1e-3))))
        t0 = time.perf_counter()
        oracle.kmeanspp(X, kk, U[-1][:kk])
        el = time.perf_counter() - t0
        result["cpu_baseline"] = {
            "value": kk / (el * k), "unit": "seedings/s", "cores": oracle.get_threads(), "kind": "oracle",
            "sample": "all %d rows of %s, the first %d of the %d draws (one pass each), scaled to k" % (
                n, w.name, kk, k)}
    return result


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed iterations (default: workload max_iters)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(
        ["blobs-10k-d16-k8", "blobs-1M-d32-k100", "aniso-8M-d16-k10", "blobs-2M-d256-k1000",
         "zipf-100M-d32-k64"]))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--full-sums", action="store_true",
                    help="recompute the sums from every point each step (KM_FLAG_FULL_SUMS)")
    ap.add_argument("--spherical", action="store_true",
                    help="spherical k-means on the same workload (KM_FLAG_SPHERICAL: rows and "
                         "centroids on the unit sphere, cosine assignment)")
    ap.add_argument("--elkan", action="store_true",
                    help="Elkan's triangle-inequality comparator (KM_FLAG_ELKAN) instead of MTI")
    ap.add_argument("--kmeanspp", action="store_true",
                    help="time k-means++ seeding of the workload's k seeds instead of the k-means steps")
    ap.add_argument("--profile", action="store_true",
                    help="run only the warmup and the timed region (no event pass, no job run, no "
                         "CPU leg), so a profiler sees warmup + K launches of each kernel")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run 5 plain device-to-device copies of 512 MiB (reference kernel "
                         "for scaling hardware byte counters)")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        nbytes = 512 << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": nbytes, "copies": 5}), flush=True)
        return 0
    if args.gpus != 1:
        print("bench.py measures the one-GPU hot path only; --gpus %d is not supported "
              "(the path runs on one GPU; the multi-GPU design is not built)" % args.gpus, file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import synth
    import paper_1902_09527_amd as km

    w = synth.WORKLOADS[args.workload]
    K = args.steps or w.max_iters
    log("workload %s: n=%d d=%d k=%d; generating" % (w.name, w.n, w.d, w.k))
    X, C0, _ = synth.make(w.name)
    if args.kmeanspp:
        print(json.dumps(bench_kmeanspp(args, w, X)), flush=True)
        return 0
    dev = torch.device("cuda:0")
    Xg = torch.from_numpy(X).to(dev)
    Cg = torch.from_numpy(C0).to(dev)
    torch.cuda.synchronize()

    # Warmup: W iterations on a throwaway context (kernel load, caches, clocks).
    if args.profile:
        args.no_cpu_baseline = True
    base_flags = {"full_sums": True} if args.full_sums else {}
    if args.spherical:
        base_flags["spherical"] = True
    if args.elkan:
        base_flags["elkan"] = True
    # profiles/<kernel>_<tag>.txt holds the counters of this workload and method
    tag = w.name + ("-spherical" if args.spherical else "") + ("-elkan" if args.elkan else "")
    if args.warmup > 0:
        with km.KMeansMTI(Xg, Cg, **base_flags) as ctx:
            for _ in range(args.warmup):
                ctx.iterate()
            torch.cuda.synchronize()
    log("warmup done (%d iterations)" % args.warmup)

    # Timed region: K iterations from C0, nothing else on the stream.
    ctx = km.KMeansMTI(Xg, Cg, **base_flags)
    path = ctx.path()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        ctx.iterate()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    hist = ctx.history()
    ctx.close()
    log("timed %d iterations in %.3f ms (path %s)" % (K, elapsed * 1e3, path))

    # The same K iterations again with HIP events around every launch (on the
    # library's stream) for the per-kernel device times; the first step is
    # timed on its own, since it runs the full streaming kernel on every path.
    def kernel_pass(**flags):
        with km.KMeansMTI(Xg, Cg, timing=True, **flags) as tctx:
            tctx.iterate()
            t_first = tctx.timing()
            for _ in range(K - 1):
                tctx.iterate()
            t_all = tctx.timing()
            h = tctx.history()
        later = {key: t_all[key] - t_first[key] for key in t_all if key.endswith("_ms")}
        return t_first, later, h

    n, d, k = w.n, w.d, w.k
    tm = first_t = later_t = None
    rooflines = []
    if not args.profile and K > 1:
        first_t, later_t, h_ev = kernel_pass(**base_flags)
        tm = {key: first_t[key] + later_t[key] for key in later_t}
        tm["iters"] = K
        kernel = DOMINANT_KERNEL.get(path, path)
        surv = n * (K - 1) - int(h_ev["clause1"][1:].sum())
        ch = int(h_ev["changed"][1:].sum())
        if path == "stream-d16":
            # Incremental steps: every point's 4-byte state read; a survivor's
            # row read and its state rewritten (Clause-1 points are not written).
            bytes_per_launch = (4 * n * (K - 1) + (4 * d + 4) * surv) / (K - 1)
            what = "steps 2..K: 4n (states) + survivors*(4d+4) (rows, new states)"
        elif path == "stream-d16-full":
            bytes_per_launch = (n * (4 * d + 4) * (K - 1) + 4 * surv) / (K - 1)
            what = "steps 2..K: n*(4d+4) (rows, states) + survivors*4 (new states)"
        elif path == "lds-elkan":
            comp = int(h_ev["computed"][1:].sum())
            bytes_per_launch = n * (4 * d + 12) + (4.0 * k * surv + 4.0 * comp + 4 * ch) / (K - 1)
            what = ("steps 2..K: n*(4d+12) + 4k per Clause-1 survivor (lower bounds read) "
                    "+ 4 per computed distance (lower bound written) + changed*4")
        else:
            bytes_per_launch = n * (4 * d + 12) + 4 * ch / (K - 1)
            what = "steps 2..K: n*(4d+12) + changed*4"
        launch_ms = later_t["assign_ms"] / (K - 1)
        flops = 2.0 * d * k * surv / (K - 1)
        if path == "global-mfma":
            # The matrix-core distance product of the survivors dominates (the
            # bound pass before it streams 8 bytes per point).
            rooflines.append(mfma_roofline_entry(kernel, tag, flops, launch_ms,
                                                 "steps 2..K: 2*d*k per Clause-1 survivor (bound pass included in the time)"))
            rooflines.append(roofline_entry(kernel, tag, bytes_per_launch, launch_ms, what))
        else:
            rooflines.append(roofline_entry(kernel, tag, bytes_per_launch, launch_ms, what))
            if path == "lds-mfma":
                rooflines.append(mfma_roofline_entry(kernel, tag, flops, launch_ms,
                                                     "steps 2..K: 2*d*k per Clause-1 survivor"))
        if path == "stream-d16":   # the full-read streaming kernel on the same steps
            _, later_f, h_f = kernel_pass(**dict(base_flags, full_sums=True))
            surv_f = n * (K - 1) - int(h_f["clause1"][1:].sum())
            rooflines.append(roofline_entry("k_small", tag, (n * (4 * d + 4) * (K - 1) + 4 * surv_f) / (K - 1),
                                            later_f["assign_ms"] / (K - 1),
                                            "steps 2..K with KM_FLAG_FULL_SUMS: n*(4d+4) + survivors*4"))

    # The job as the workload defines it (tol stop), for the iteration count.
    job = {"iterations": 0, "converged": 0, "device_ms": 0.0}
    if not args.profile:
        _, _, job = km.run(Xg, Cg, w.max_iters, w.tol, **base_flags)
        torch.cuda.synchronize()

    ips = K / elapsed
    computed = int(hist["computed"].sum())
    lloyd = n * k * K
    roof = rooflines[0] if rooflines else {"kernel": DOMINANT_KERNEL.get(path, path), "bound": "hbm",
                                          "achieved": None, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                          "frac": None, "traffic": None}
    result = {
        "metric": METRIC,
        "value": ips,
        "unit": "iters/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "method": ("spherical" if args.spherical else "kmeans") +
                   ("+elkan-ti" if args.elkan else ""),
                   "n": n, "d": d, "k": k, "max_iters": w.max_iters, "tol": w.tol,
                   "timed": "first %d iterations from the seeded centroids" % K, "path": path},
        "eff_dist_evals_per_s": lloyd / elapsed,
        # The bytes a full-read Lloyd step moves (every row and its point
        # state) over the measured step time, against the HBM peak: above 1
        # when pruning skips rows.
        "full_read_equiv_hbm_frac": n * (4 * d + 4) / (elapsed / K) / (HBM_PEAK_GBS * 1e9),
        "computed_dist_evals_per_s": computed / elapsed,
        "pruned_frac": 1.0 - computed / lloyd,
        "clause1_frac": float(hist["clause1"].sum()) / (n * K),
        "kernel_ms_per_iter": None if tm is None else
            {key[:-3]: tm[key] / max(1, tm["iters"]) for key in ("assign_ms", "reduce_ms", "update_ms", "table_ms")},
        "first_step_ms": None if first_t is None else
            {key[:-3]: first_t[key] for key in ("assign_ms", "reduce_ms", "update_ms", "table_ms")},
        "job": {"iterations": job["iterations"], "converged": bool(job["converged"]),
                "device_ms": job["device_ms"],
                "iters_per_s": job["iterations"] / (job["device_ms"] / 1e3) if job["device_ms"] else None},
        "roofline": roof,
        "rooflines_all": rooflines[1:],
    }
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        result["cpu_baseline"] = cpu_baseline(X, C0, w, spherical=args.spherical)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
