"""Elkan's triangle-inequality comparator (KM_FLAG_ELKAN) on the GPU.

Elkan's pruning is exact, so its results are the oracle's (plain float64
Lloyd's) and bitwise those of the MTI kernels on the same inputs; what
differs is the work: a lower bound per point and centroid prunes more
distances (the paper's comparison of MTI with TI, section III-C and the MTI
evaluation), at O(nk) memory.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from parity import check_assign, check_centroids

import paper_1902_09527_amd as km
from paper_1902_09527_amd import _native as N

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _gpu(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(DEV)


CASES = [
    # seed, n, d, k, spread, sigma, iters, tol
    (401, 5000 + 7, 16, 10, 3.0, 1.0, 20, 0.0),
    (402, 3 * 256 + 37, 32, 20, 5.0, 2.0, 25, 0.0),
    (403, 5000, 3, 7, 4.0, 1.5, 30, 0.0),
    (404, 2000, 1, 5, 3.0, 1.0, 20, 0.0),
    (405, 4000, 16, 1, 3.0, 1.0, 5, 0.0),
    (406, 3000, 5, 50, 3.0, 1.0, 40, 0.001),
    (407, 4096 + 1, 64, 30, 5.0, 2.0, 15, 0.0),
    (408, 20000, 32, 100, 20.0, 1.5, 30, 0.0),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "s%d-n%d-d%d-k%d" % c[:4])
def test_elkan_matches_oracle_and_mti(case):
    seed, n, d, k, spread, sigma, iters, tol = case
    print("case", case, flush=True)
    X, C0 = synth.blobs(n, d, k, seed=seed, spread=spread, sigma=sigma)
    ref = oracle.lloyd(X, C0, iters, tol)
    Xg, Cg = _gpu(X), _gpu(C0)
    with km.KMeansMTI(Xg, Cg, elkan=True) as ctx:
        assert ctx.path() == "lds-elkan"
    a, c, st = km.run(Xg, Cg, iters, tol, elkan=True, stats=True)
    assert st["iterations"] == ref["iters"]
    check_assign(a.cpu().numpy(), ref["assign"], ref["best"], ref["second"], "final assignment")
    check_centroids(c.cpu().numpy(), ref["C"], X, "final centroids")
    assert st["inertia_last"] == pytest.approx(ref["inertia"][-1], rel=1e-5)
    # the same exact decisions as the MTI vector scan: bitwise equal outputs
    a2, c2, st2 = km.run(Xg, Cg, iters, tol, generic=True, vector_only=True)
    assert torch.equal(a, a2) and torch.equal(c, c2)
    assert st["iterations"] == st2["iterations"]
    assert st["dist_computed"] <= st["dist_lloyd"]


def test_elkan_trajectory_and_no_prune():
    X, C0 = synth.blobs(30000 + 5, 24, 40, seed=409, spread=4.0, sigma=1.5)
    T = 12
    ref = oracle.lloyd(X, C0, T, history=True)
    Xg, Cg = _gpu(X), _gpu(C0)
    with km.KMeansMTI(Xg, Cg, elkan=True) as ctx:
        for t in range(T):
            print("step", t, flush=True)
            ch = ctx.iterate(sync=True)
            a, c = ctx.get()
            prev = None if t == 0 else ref["assign_hist"][t - 1]
            _, b, s, _ = oracle.assign(X, ref["C_hist"][t], prev=prev)
            info = check_assign(a.cpu().numpy(), ref["assign_hist"][t], b, s, "step %d" % t)
            if info["mismatch"] == 0:
                assert ch == ref["changed"][t]
            np.testing.assert_allclose(ctx.centroids64(), ref["C_hist"][t + 1], rtol=1e-9, atol=1e-9)
    a1, c1, _ = km.run(Xg, Cg, T, elkan=True)
    a0, c0, s0 = km.run(Xg, Cg, T, elkan=True, prune=False)
    assert torch.equal(a1, a0) and torch.equal(c1, c0)
    assert s0["dist_computed"] == X.shape[0] * 40 * T


def test_elkan_prunes_at_least_as_much_as_mti_on_clustered_data():
    # the lower bounds can only add skips to the same scan; lazily tightened
    # bounds may fail MTI's whole-point test more often, but on clustered
    # data the per-centroid bounds win by a wide margin
    X, C0 = synth.blobs(200000 + 3, 32, 64, seed=410, spread=10.0, sigma=1.0)
    Xg, Cg = _gpu(X), _gpu(C0)
    _, _, ti = km.run(Xg, Cg, 20, elkan=True)
    _, _, mti = km.run(Xg, Cg, 20, generic=True, vector_only=True)
    print("computed TI", ti["dist_computed"], "MTI", mti["dist_computed"], flush=True)
    assert ti["dist_computed"] < mti["dist_computed"]


def test_elkan_refuses_the_global_path():
    X, C0 = synth.blobs(4000 + 3, 256, 1000, seed=411)
    with pytest.raises(N.KMError) as e:
        km.KMeansMTI(_gpu(X), _gpu(C0), elkan=True)
    assert e.value.status == N.KM_ERR_UNSUPPORTED
    X, C0 = synth.blobs(1000, 16, 10, seed=412)
    with pytest.raises(N.KMError) as e:
        km.KMeansMTI(_gpu(X), _gpu(C0), elkan=True, large_path=True)
    assert e.value.status == N.KM_ERR_INVALID_ARG


def test_elkan_full_size_workload_equals_mti():
    X, C0, w = synth.make("blobs-1M-d32-k100")
    Xg, Cg = _gpu(X), _gpu(C0)
    a1, c1, s1 = km.run(Xg, Cg, w.max_iters, w.tol, elkan=True)
    a2, c2, s2 = km.run(Xg, Cg, w.max_iters, w.tol, generic=True, vector_only=True)
    assert torch.equal(a1, a2) and torch.equal(c1, c2)
    assert s1["iterations"] == s2["iterations"]
    print("computed TI", s1["dist_computed"], "MTI", s2["dist_computed"], flush=True)
