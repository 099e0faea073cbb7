#!/usr/bin/env python3
"""Write whole-run oracle digests of the two largest workloads.

    python tests/golden/make_workload_digests.py [NAME ...]

For each workload (default: blobs-2M-d256-k1000 and zipf-100M-d32-k64) this
runs the plain float64 Lloyd's oracle (oracle.lloyd: no pruning, section IV-A)
once over all rows from the seeded initial centroids, for the workload's
max_iters and tol, and stores what a GPU run must reproduce:

  workload_<name>.json
      iterations, per-step changed counts and inertia, final cluster sizes,
      the rows whose final best-vs-second relative gap (D2 - D1) / D2 of
      squared distances is <= 1e-5 (near ties, where the assignment is not
      required to match), and the SHA-256 of the final int32 assignment
      (little-endian) with those rows set to -1;
  workload_<name>_C.npy
      the final float64 centroids (k x d).

Inputs come from synth.make(name); nothing else is read.  Only oracle/ and
synth/ are called.  Runs on the host's cores (OpenMP); a run of the 2M x 256,
k = 1000 workload takes on the order of 20 minutes on 8 cores.
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import synth  # noqa: E402

GAP = 1e-5
DEFAULT = ["blobs-2M-d256-k1000", "zipf-100M-d32-k64"]


def near_tie_rows(best: np.ndarray, second: np.ndarray) -> np.ndarray:
    """Rows whose relative gap (second - best) / second is <= GAP (gap 0 when second is 0)."""
    with np.errstate(divide="ignore", invalid="ignore"):
        g = (second - best) / second
    g = np.where(np.isinf(second), 1.0, g)
    g = np.where(second == 0, 0.0, g)
    return np.nonzero(g <= GAP)[0].astype(np.int64)


def masked_hash(assign: np.ndarray, ties: np.ndarray) -> str:
    a = np.ascontiguousarray(assign, dtype="<i4").copy()
    a[ties] = -1
    return hashlib.sha256(a.tobytes()).hexdigest()


def digest(name: str) -> None:
    t0 = time.time()
    X, C0, w = synth.make(name)
    print("[digest] %s: generated %d x %d in %.0f s" % (name, w.n, w.d, time.time() - t0), flush=True)
    t0 = time.time()
    ref = oracle.lloyd(X, C0, w.max_iters, w.tol)
    el = time.time() - t0
    print("[digest] %s: oracle %d iterations in %.0f s on %d threads" % (
        name, ref["iters"], el, oracle.get_threads()), flush=True)
    ties = near_tie_rows(ref["best"], ref["second"])
    counts = np.bincount(ref["assign"], minlength=w.k).astype(np.int64)
    rec = {
        "workload": name, "n": w.n, "d": w.d, "k": w.k, "max_iters": w.max_iters, "tol": w.tol,
        "source": "tests/golden/make_workload_digests.py: oracle.lloyd (plain float64 Lloyd's, "
                  "section IV-A) on synth.make(%r), all rows, from the seeded initial centroids" % name,
        "iterations": int(ref["iters"]),
        "changed": [int(v) for v in ref["changed"]],
        "inertia": [float(v) for v in ref["inertia"]],
        "counts": [int(v) for v in counts],
        "gap": GAP,
        "near_tie_rows": [int(v) for v in ties],
        "assign_sha256_ties_masked": masked_hash(ref["assign"], ties),
        "oracle_seconds": round(el, 1),
        "oracle_threads": oracle.get_threads(),
    }
    with open(os.path.join(HERE, "workload_%s.json" % name), "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    np.save(os.path.join(HERE, "workload_%s_C.npy" % name), np.ascontiguousarray(ref["C"], np.float64))
    print("[digest] %s: %d near ties, changed %s" % (name, len(ties), rec["changed"]), flush=True)


def main(argv) -> int:
    for name in argv or DEFAULT:
        digest(name)
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
