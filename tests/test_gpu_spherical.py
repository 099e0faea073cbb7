"""Spherical k-means (KM_FLAG_SPHERICAL) on every kernel path against the
float64 spherical oracle, through the C ABI.

The oracle works from the raw rows with exact cosines; the GPU projects the
rows to the unit sphere once (float64 norm, float32 unit rows) and runs the
Euclidean machinery on them, so the comparison rules are those of k-means
with the oracle's squared chord distances 2 - 2 cos as the best/second
distances and unit vectors as the scale of the centroid error.
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


def _unit(A):
    A = np.asarray(A, np.float64)
    r = np.linalg.norm(A, axis=1, keepdims=True)
    return np.where(r > 0, A / np.where(r > 0, r, 1.0), 0.0)


CASES = [
    # seed, n, d, k, spread, sigma, iters, tol, flags, path
    (201, 5000 + 3, 16, 10, 3.0, 1.0, 20, 0.0, {}, "stream-d16"),
    (202, 40000 + 11, 16, 16, 2.0, 1.5, 25, 0.0, {}, "stream-d16"),
    (203, 20000 + 7, 16, 7, 3.0, 1.0, 20, 0.001, {"stats": True}, "stream-d16-full"),
    (204, 3000 + 1, 5, 7, 3.0, 1.0, 25, 0.0, {"stats": True}, "lds-vector"),
    (205, 6000 + 5, 32, 40, 4.0, 2.0, 20, 0.0, {"stats": True}, "lds-mfma"),
    (206, 5000, 64, 200, 6.0, 2.0, 12, 0.0, {"stats": True}, "global-mfma"),
    (207, 4000 + 3, 64, 50, 3.0, 1.0, 10, 0.0, {"large_path": True, "stats": True}, "global-mfma"),
    (208, 3000, 16, 12, 3.0, 1.0, 15, 0.0, {"generic": True, "stats": True}, "lds-vector"),
    (209, 6000 + 5, 32, 40, 4.0, 2.0, 20, 0.0, {}, "lds-inc"),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "s%d-n%d-d%d-k%d" % c[:4])
def test_spherical_matches_oracle(case):
    seed, n, d, k, spread, sigma, iters, tol, flags, path = case
    print("case", case[:8], flags, flush=True)
    X, C0 = synth.blobs(n, d, k, seed=seed, spread=spread, sigma=sigma)
    ref = oracle.spherical(X, C0, iters, tol)
    with km.KMeansMTI(_gpu(X), _gpu(C0), spherical=True, **flags) as ctx:
        assert ctx.path() == path
    a, c, st = km.run(_gpu(X), _gpu(C0), iters, tol, spherical=True, **flags)
    assert st["iterations"] == ref["iters"]
    check_assign(a.cpu().numpy(), ref["assign"], ref["best"], ref["second"], "final assignment")
    c = c.cpu().numpy()
    check_centroids(c, ref["C"], _unit(X), "final centroids")
    np.testing.assert_allclose(np.linalg.norm(c.astype(np.float64), axis=1), 1.0, rtol=0, atol=1e-6)
    if flags.get("stats"):
        assert st["inertia_last"] == pytest.approx(ref["objective"][-1], rel=1e-4)


@pytest.mark.parametrize("stats", [False, True], ids=["incremental", "full+inertia"])
def test_spherical_every_step_matches_oracle(stats):
    # the assignment, changed count and centroids after every step, each
    # against an oracle run of that many steps
    X, C0 = synth.blobs(30000 + 17, 16, 9, seed=209, spread=2.0, sigma=1.5)
    T = 12
    with km.KMeansMTI(_gpu(X), _gpu(C0), spherical=True, stats=stats) as ctx:
        assert ctx.path() == ("stream-d16-full" if stats else "stream-d16")
        for t in range(T):
            print("step", t, flush=True)
            ch = ctx.iterate(sync=True)
            a, c = ctx.get()
            ref = oracle.spherical(X, C0, t + 1)
            info = check_assign(a.cpu().numpy(), ref["assign"], ref["best"], ref["second"], "step %d" % t)
            if info["mismatch"] == 0:
                assert ch == ref["changed"][t]
            check_centroids(c.cpu().numpy(), ref["C"], _unit(X), "step %d" % t, tol=1e-6)
            if stats:
                assert ctx.history()["inertia"][t] == pytest.approx(ref["objective"][t], rel=1e-4)


def test_spherical_prune_and_no_prune_are_bitwise_identical():
    X, C0 = synth.blobs(20000 + 9, 16, 10, seed=210, spread=2.0, sigma=1.0)
    Xg, Cg = _gpu(X), _gpu(C0)
    a1, c1, s1 = km.run(Xg, Cg, 20, spherical=True, prune=True)
    a2, c2, s2 = km.run(Xg, Cg, 20, spherical=True, prune=False)
    assert torch.equal(a1, a2) and torch.equal(c1, c2)
    assert s1["iterations"] == s2["iterations"]


def test_spherical_power_of_two_row_scaling_is_bitwise_invisible():
    # x * 2^e has the same float64 unit vector, hence the same float32 unit
    # row: a size the oracle is not run at, checked by an exact invariance.
    X, C0 = synth.blobs(1_000_000 + 21, 16, 10, seed=211, spread=3.0, sigma=1.0)
    rng = np.random.default_rng(211)
    e = rng.integers(-30, 30, size=(X.shape[0], 1)).astype(np.float64)
    Xs = (X.astype(np.float64) * 2.0 ** e).astype(np.float32)
    a1, c1, s1 = km.run(_gpu(X), _gpu(C0), 12, spherical=True)
    a2, c2, s2 = km.run(_gpu(Xs), _gpu(C0 * 4.0), 12, spherical=True)
    assert torch.equal(a1, a2) and torch.equal(c1, c2)
    assert s1["iterations"] == s2["iterations"]


def test_spherical_zero_rows_and_zero_centroid():
    X, C0 = synth.blobs(2000, 16, 6, seed=212, spread=2.0)
    X = X.copy()
    X[[3, 700, 1999]] = 0.0
    ref = oracle.spherical(X, C0, 10)
    a, c, st = km.run(_gpu(X), _gpu(C0), 10, spherical=True)
    a = a.cpu().numpy()
    check_assign(a, ref["assign"], ref["best"], ref["second"], "final assignment")
    check_centroids(c.cpu().numpy(), ref["C"], _unit(X), "final centroids")
    assert (a[[3, 700, 1999]] >= 0).all() and (a[[3, 700, 1999]] < 6).all()
    C0z = C0.copy()
    C0z[4] = 0.0
    with pytest.raises(N.KMError) as ei:
        km.run(_gpu(X), _gpu(C0z), 3, spherical=True)
    assert ei.value.status == N.KM_ERR_INVALID_ARG
