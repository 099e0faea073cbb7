"""The five benchmark workloads on the GPU, checked against the CPU oracle.

The three smaller workloads run whole on both sides (assignments except
oracle near ties, centroids, iteration count).  The 100M-point and the
2M x 256, k = 1000 workloads are too large for a whole oracle run; there
every checked step is compared at full size in the launch configuration the
benchmark uses: the oracle's assignment step on a seeded sample of points,
from the GPU's own float64 centroids and previous assignment, and the
oracle's update step over all points from the GPU's assignment.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from parity import check_assign, check_centroids

import paper_1902_09527_amd as km

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _whole(name):
    X, C0, w = synth.make(name)
    print("workload", name, flush=True)
    ref = oracle.lloyd(X, C0, w.max_iters, w.tol)
    a, c, st = km.run(torch.from_numpy(X).cuda(), torch.from_numpy(C0).cuda(), w.max_iters, w.tol)
    torch.cuda.synchronize()
    assert st["iterations"] == ref["iters"]
    info = check_assign(a.cpu().numpy(), ref["assign"], ref["best"], ref["second"], name)
    err = check_centroids(c.cpu().numpy(), ref["C"], X, name)
    print(name, "iterations", st["iterations"], "mismatches", info, "centroid rel err %.2e" % err,
          flush=True)


@pytest.mark.parametrize("name", ["blobs-10k-d16-k8", "blobs-1M-d32-k100", "aniso-8M-d16-k10"])
def test_workload_whole_run(name):
    _whole(name)


@pytest.mark.parametrize("name,sample", [("zipf-100M-d32-k64", 1_000_000), ("blobs-2M-d256-k1000", 20_000)])
def test_large_workload_steps_sampled(name, sample):
    X, C0, w = synth.make(name)
    print("generated", name, flush=True)
    n = w.n
    rng = np.random.default_rng(2024)
    sample = np.sort(rng.choice(n, sample, replace=False))
    Xs = np.ascontiguousarray(X[sample])
    check_at = {0, 1, w.max_iters - 1}
    with km.KMeansMTI(torch.from_numpy(X).cuda(), torch.from_numpy(C0).cuda()) as ctx:
        prev = None
        for t in range(w.max_iters):
            C_before = ctx.centroids64() if t in check_at else None
            ctx.iterate()
            if t in check_at or t + 1 in check_at:
                a, _ = ctx.get(centroids=False)
                a = a.cpu().numpy()
            if t in check_at:
                pv = None if prev is None else prev[sample]
                ra, rb, rs, _ = oracle.assign(Xs, C_before, prev=pv)
                info = check_assign(a[sample], ra, rb, rs, "step %d (sample)" % t)
                C_ref, counts = oracle.update(X, a, C_before)
                assert counts.sum() == n
                err = check_centroids(ctx.centroids64(), C_ref, X[:100_000], "step %d" % t)
                print("step", t, info, "centroid rel err %.2e" % err, flush=True)
            prev = a if (t + 1 in check_at) else None
