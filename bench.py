#!/usr/bin/env python3
"""Benchmark of the MTI k-means hot path on one MI355X.

An iteration is one Lloyd step with MTI pruning: centroid table and drift,
bound update and Clause-1 test, fused distance + argmin of the survivors,
per-cluster reduction into new centroids and the convergence counters.  A
timed step is one whole run of the workload as it is defined: a
kmeans_mti_run call from the seeded initial centroids until fewer than
tol * n points change assignment (or max_iters), context set-up and release
included, with the inputs already resident in HBM.  K runs are timed between
device synchronisations; the reported value is iterations per second over
them.  The steady state (steps after the first) and the first step are
reported beside it from HIP events the library records on its stream around
every launch.

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
MFMA_BF16_PEAK_TFS = 2500.0  # MI355X dense bf16 matrix peak (the split products of k_mfma_large, k_inc_mm)
DEFAULT_WORKLOAD = "aniso-8M-d16-k10"
METRIC = "k-means iters/sec + effective dist evals/sec; % HBM peak (low d) / % MFMA (big k·d)"


def log(msg: str) -> None:
    print("[bench] " + msg, file=sys.stderr, flush=True)


# Dominant (assignment-step) kernel of each library path.
DOMINANT_KERNEL = {"stream-d16": "k_inc", "stream-d16-full": "k_small", "lds-vector": "k_assign",
                   "lds-mfma": "k_assign", "lds-elkan": "k_assign", "lds-inc": "k_inc_mm",
                   "global-mfma": "k_mfma_large"}
# Sources of each dominant kernel: the hardware byte counts of a committed
# profile summary are used only while these files are unchanged.
# km_capi.hip sets each kernel's grid and LDS, so it is part of every hash.
KERNEL_SOURCES = {
    "k_small": ["km_small.hip", "km_device.h", "km_internal.h", "km_capi.hip"],
    "k_inc": ["km_small.hip", "km_device.h", "km_internal.h", "km_capi.hip"],
    "k_first": ["km_small.hip", "km_device.h", "km_internal.h", "km_capi.hip"],
    "k_assign": ["km_kernels.hip", "km_device.h", "km_internal.h", "km_capi.hip"],
    "k_inc_mm": ["km_incmm.hip", "km_device.h", "km_internal.h", "km_capi.hip"],
    "k_mfma_large": ["km_large.hip", "km_device.h", "km_internal.h", "km_capi.hip"],
    "k_pp_step": ["km_pp.hip", "km_device.h", "km_internal.h", "km_capi.hip"],
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
                        what: str, peak: float = MFMA_F32_PEAK_TFS, dtype: str = "f32") -> dict:
    """Matrix-core roofline of one kernel: algorithmic flops per launch over its
    mean launch time (HIP events), against the dense peak of the products'
    dtype."""
    achieved = flops_per_launch / (launch_ms / 1e3) / 1e12
    traffic, source = measured_traffic(kernel, workload)
    return {"kernel": kernel, "bound": "mfma", "achieved": achieved, "peak": peak,
            "unit": "TFLOP/s", "frac": achieved / peak, "traffic": traffic, "mfma_dtype": dtype,
            "traffic_source": source, "flops_per_launch": flops_per_launch, "flops_def": what,
            "kernel_us": launch_ms * 1e3}


def host_cpu() -> dict:
    """CPU model and the cores this process may use."""
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
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count() or 1
    return {"cpu_model": model, "nproc": nproc}


def cpu_baseline(X, C0, w, spherical: bool = False) -> dict:
    """Time the CPU oracle as it stands on this host: plain float64 Lloyd's
    on every thread OpenMP gives it (value), on one thread, and the float64
    MTI reference on every thread (the paper's method on the host).  Each leg
    is bounded to about 10 s of CPU work and scaled to iterations/s."""
    import oracle
    if spherical:   # the spherical oracle is a single-threaded loop
        t0 = time.perf_counter()
        r = oracle.spherical(X, C0, 1, 0.0)
        t1 = time.perf_counter() - t0
        iters = int(max(1, min(w.max_iters, 10.0 // max(t1, 1e-3))))
        t0 = time.perf_counter()
        r = oracle.spherical(X, C0, iters, w.tol)
        el = time.perf_counter() - t0
        return dict(host_cpu(), value=r["iters"] / el, unit="iters/s", cores=1, kind="oracle",
                    sample="all %d rows of %s, spherical k-means run from the seeded centroids "
                           "(tol %g), first %d iterations" % (w.n, w.name, w.tol, r["iters"]))
    P = oracle.get_threads()
    t0 = time.perf_counter()
    oracle.lloyd(X, C0, 1, 0.0)
    t1 = time.perf_counter() - t0
    # P threads: the workload's own run (tol stop), at most ~10 s of iterations
    cap = int(max(1, min(w.max_iters, 10.0 // max(t1, 1e-3))))
    t0 = time.perf_counter()
    r = oracle.lloyd(X, C0, cap, w.tol)
    el = time.perf_counter() - t0
    out = dict(host_cpu(), value=r["iters"] / el, unit="iters/s", cores=P, kind="oracle",
               sample="all %d rows of %s, the run from the seeded centroids with tol %g: %d iterations%s "
                      "(%.3g effective dist evals/s)" % (
                          w.n, w.name, w.tol, r["iters"],
                          " (capped)" if r["iters"] == cap and cap < w.max_iters else "",
                          r["iters"] * w.n * w.k / el))
    # one thread: one iteration on a row prefix sized to ~10 s, scaled to all rows
    rows = int(min(w.n, max(w.k, w.n * 10.0 / max(t1 * P, 1e-3))))
    oracle.set_threads(1)
    try:
        t0 = time.perf_counter()
        oracle.lloyd(X[:rows], C0, 1, 0.0)
        el1 = time.perf_counter() - t0
    finally:
        oracle.set_threads(P)
    out["one_thread"] = {"value": rows / (el1 * w.n), "unit": "iters/s", "cores": 1,
                         "sample": "first iteration on the first %d rows, scaled to %d rows" % (rows, w.n)}
    # the float64 MTI reference (pruned Lloyd's on the host) on P threads
    t0 = time.perf_counter()
    rm = oracle.mti(X, C0, cap, w.tol)
    elm = time.perf_counter() - t0
    out["mti_ref"] = {"value": rm["iters"] / elm, "unit": "iters/s", "cores": P,
                      "pruned_frac": 1.0 - float(rm["computed"].sum()) / (w.n * w.k * rm["iters"]),
                      "sample": "the same run with the float64 MTI reference (%d iterations)" % rm["iters"]}
    return out


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
    ap.add_argument("--steps", type=int, default=None,
                    help="timed whole runs of the workload (default 20; k-means++: seedings, default 5)")
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
                    help="for a profiler: the warmup runs, then K contexts that each run exactly the "
                         "workload's T iterations (no launches past the stop, no event pass, no CPU "
                         "leg); prints T and the path")
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
    K = args.steps or 20
    if args.profile:
        args.no_cpu_baseline = True
    log("workload %s: n=%d d=%d k=%d; generating" % (w.name, w.n, w.d, w.k))
    X, C0, _ = synth.make(w.name)
    if args.kmeanspp:
        print(json.dumps(bench_kmeanspp(args, w, X)), flush=True)
        return 0
    dev = torch.device("cuda:0")
    Xg = torch.from_numpy(X).to(dev)
    Cg = torch.from_numpy(C0).to(dev)
    torch.cuda.synchronize()

    base_flags = {"full_sums": True} if args.full_sums else {}
    if args.spherical:
        base_flags["spherical"] = True
    if args.elkan:
        base_flags["elkan"] = True
    # profiles/<kernel>_<tag>.txt holds the counters of this workload and method
    tag = w.name + ("-spherical" if args.spherical else "") + ("-elkan" if args.elkan else "")

    def job():
        return km.run(Xg, Cg, w.max_iters, w.tol, **base_flags)

    # Warmup: W whole runs (kernel load, caches, clocks).
    for _ in range(args.warmup):
        job()
    torch.cuda.synchronize()
    log("warmup done (%d runs)" % args.warmup)

    if args.profile:
        # K contexts of exactly the run's T steps: each kernel's dispatches
        # are then T per context (the first step first), in order.
        T = job()[2]["iterations"]
        torch.cuda.synchronize()
        for _ in range(K):
            with km.KMeansMTI(Xg, Cg, **base_flags) as pctx:
                path = pctx.path()
                for _ in range(T):
                    pctx.iterate()
                pctx.get()
        torch.cuda.synchronize()
        print(json.dumps({"profile": True, "workload": w.name, "contexts": K, "iterations": T, "path": path}),
              flush=True)
        return 0

    # Timed region: K whole runs of the workload as it is defined (from the
    # seeded centroids until fewer than tol * n points change, or max_iters),
    # each a kmeans_mti_run call: context set-up, iterations, results, release.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    runs = [job()[2] for _ in range(K)]
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    iters = runs[0]["iterations"]
    assert all(r["iterations"] == iters for r in runs), "runs differ in their iteration count"
    loop_ms = sum(r["device_ms"] for r in runs) / K
    n, d, k = w.n, w.d, w.k
    with km.KMeansMTI(Xg, Cg, **base_flags) as pctx:
        path = pctx.path()
    log("timed %d runs of %d iterations in %.3f ms (path %s)" % (K, iters, elapsed * 1e3, path))

    # The same run's iterations again with HIP events around every launch (on
    # the library's stream): the first step on its own, then steps 1..T-1 as
    # the steady state.
    def kernel_pass(T, **flags):
        with km.KMeansMTI(Xg, Cg, timing=True, **flags) as tctx:
            tctx.iterate()
            t_first = tctx.timing()
            for _ in range(T - 1):
                tctx.iterate()
            t_all = tctx.timing()
            h = tctx.history()
        later = {key: t_all[key] - t_first[key] for key in t_all if key.endswith("_ms")}
        return t_first, later, h

    KS = max(iters, 2)   # steps of the steady-state pass (a one-step run adds one step)
    first_t = later_t = None
    rooflines = []
    steady = None
    hist = None
    if not args.profile:
        first_t, later_t, hist = kernel_pass(KS, **base_flags)
        m = KS - 1
        steady_ms = sum(later_t[key] for key in ("assign_ms", "reduce_ms", "update_ms", "table_ms")) / m
        steady = {"steps": "1..%d" % (KS - 1), "ms_per_iter": steady_ms, "iters_per_s": 1e3 / steady_ms,
                  "kernel_ms_per_iter": {key[:-3]: later_t[key] / m for key in
                                         ("assign_ms", "reduce_ms", "update_ms", "table_ms")}}
        kernel = DOMINANT_KERNEL.get(path, path)
        surv = n * m - int(hist["clause1"][1:KS].sum())
        ch = int(hist["changed"][1:KS].sum())
        comp = int(hist["computed"][1:KS].sum())
        launch_ms = later_t["assign_ms"] / m
        # Algorithmic bytes per step: every point's assignment read and bound
        # read and written (12 B) plus, with incremental sums, the rows of the
        # Clause-1 survivors and of the changed points (4d B each), or with
        # full sums every row (4d B) and the changed assignments (4 B).
        if path in ("stream-d16", "lds-inc"):
            bytes_per_launch = 12.0 * n + 4.0 * d * (surv + ch) / m
            what = "steps 1..T-1: 12n (assignment, bound) + 4d per Clause-1 survivor and per changed point"
        elif path == "lds-elkan":
            bytes_per_launch = n * (4 * d + 12) + (4.0 * k * surv + 4.0 * comp + 4 * ch) / m
            what = ("steps 1..T-1: n*(4d+12) + 4k per Clause-1 survivor (lower bounds read) "
                    "+ 4 per computed distance (lower bound written) + changed*4")
        else:
            bytes_per_launch = n * (4 * d + 12) + 4.0 * ch / m
            what = "steps 1..T-1: n*(4d+12) (rows, assignment, bound) + changed*4"
        flops = 2.0 * d * k * surv / m
        if path == "lds-inc":   # the dense products of the centroid blocks evaluated
            flops = 2.0 * d * comp / m
        if path == "global-mfma":
            rooflines.append(mfma_roofline_entry(kernel, tag, flops, launch_ms,
                                                 "steps 1..T-1: 2*d*k per Clause-1 survivor (bound pass included "
                                                 "in the time); the matrix cores run 3 bf16 products per dot "
                                                 "(3x these flops)", MFMA_BF16_PEAK_TFS, "bf16"))
            rooflines.append(roofline_entry(kernel, tag, bytes_per_launch, launch_ms, what))
        else:
            rooflines.append(roofline_entry(kernel, tag, bytes_per_launch, launch_ms, what))
            if path == "lds-mfma":
                rooflines.append(mfma_roofline_entry(kernel, tag, flops, launch_ms,
                                                     "steps 1..T-1: 2*d*k per Clause-1 survivor"))
            if path == "lds-inc":
                rooflines.append(mfma_roofline_entry(kernel, tag, flops, launch_ms,
                                                     "steps 1..T-1: 2*d per distance of the evaluated "
                                                     "32-centroid blocks; the matrix cores run 3 bf16 "
                                                     "products per dot (3x these flops)", MFMA_BF16_PEAK_TFS,
                                                     "bf16"))
        if path == "stream-d16":   # the full-read streaming kernel on the same steps
            _, later_f, h_f = kernel_pass(KS, **dict(base_flags, full_sums=True))
            ch_f = int(h_f["changed"][1:KS].sum())
            rooflines.append(roofline_entry("k_small", tag, n * (4 * d + 12) + 4.0 * ch_f / m,
                                            later_f["assign_ms"] / m,
                                            "steps 1..T-1 with KM_FLAG_FULL_SUMS: n*(4d+12) + changed*4"))
        # The first step (no bounds yet): every row read and every point's
        # assignment and bound written; on the global path every point's k
        # distances go through the matrix cores.
        # (the stream path's first step runs in k_first unless statistics are gathered)
        first_kernel = "k_first" if path.startswith("stream") else kernel
        if path == "global-mfma":
            rooflines.append(mfma_roofline_entry(first_kernel, tag + "-first-step", 2.0 * d * k * n,
                                                 first_t["assign_ms"], "first step: 2*d*k per point (3 bf16 "
                                                 "products per dot)", MFMA_BF16_PEAK_TFS, "bf16"))
        else:
            rooflines.append(roofline_entry(first_kernel, tag + "-first-step", n * (4.0 * d + 8),
                                            first_t["assign_ms"],
                                            "first step: n*(4d+8) (rows read, assignment and bound written)"))

    value = K * iters / elapsed
    lloyd = n * k * KS
    roof = rooflines[0] if rooflines else {"kernel": DOMINANT_KERNEL.get(path, path), "bound": "hbm",
                                          "achieved": None, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                          "frac": None, "traffic": None}
    result = {
        "metric": METRIC,
        "value": value,
        "unit": "iters/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16x3+f32" if path in ("global-mfma", "lds-inc") else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "method": ("spherical" if args.spherical else "kmeans") +
                   ("+elkan-ti" if args.elkan else ""),
                   "n": n, "d": d, "k": k, "max_iters": w.max_iters, "tol": w.tol,
                   "step": "one whole run (kmeans_mti_run from the seeded centroids to the tol stop, "
                           "set-up and release included)",
                   "iters_per_step": iters, "converged": bool(runs[0]["converged"]), "path": path},
        "ms_per_iter": elapsed * 1e3 / (K * iters),
        "eff_dist_evals_per_s": value * n * k,
        "run_loop_device_ms": loop_ms,
        "run_setup_ms": elapsed * 1e3 / K - loop_ms,
        "steady_state": steady,
        "first_step_ms": None if first_t is None else
            {key[:-3]: first_t[key] for key in ("assign_ms", "reduce_ms", "update_ms", "table_ms")},
        "roofline": roof,
        "rooflines_all": rooflines[1:],
    }
    if hist is not None:
        computed = int(hist["computed"][:KS].sum())
        result.update({
            "computed_dist_evals_per_s": value * computed / KS,
            "pruned_frac": 1.0 - computed / lloyd,
            "pruned_frac_steady": 1.0 - int(hist["computed"][1:KS].sum()) / (n * k * (KS - 1)),
            "clause1_frac_steady": float(hist["clause1"][1:KS].sum()) / (n * (KS - 1)),
        })
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        result["cpu_baseline"] = cpu_baseline(X, C0, w, spherical=args.spherical)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
