"""The incremental matrix-core path ("lds-inc": d = 16 or 32, k <= 128) on the
GPU, through the C ABI.

It reads only the Clause-1 survivors' rows after the first step and moves
the rows of the points whose cluster changed between exact integer sums, so
it must give bitwise the results of the full-read path (KM_FLAG_FULL_SUMS:
every row added each step) and the oracle's results.  Sizes span several
256-point wave tiles with a ragged tail, fewer tiles than waves, one and
several centroid blocks of 32 with padded blocks (k = 1, 17, 33, 65, 100,
128).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from parity import check_assign, check_centroids

import paper_1902_09527_amd as km

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _gpu(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(DEV)


CASES = [
    # seed, n, d, k, spread, sigma, iters, tol
    (501, 8 * 256 * 3 + 37, 32, 100, 20.0, 1.5, 20, 0.0),
    (502, 5000 + 3, 16, 17, 4.0, 2.0, 20, 0.0),
    (503, 300, 32, 1, 3.0, 1.0, 5, 0.0),
    (504, 20000 + 11, 32, 33, 6.0, 2.0, 25, 0.001),
    (505, 12000 + 5, 16, 65, 3.0, 1.5, 20, 0.0),
    (506, 30000 + 1, 32, 128, 10.0, 2.0, 15, 0.0),
    (507, 777, 32, 10, 5.0, 2.0, 20, 0.0),
    (508, 60000 + 13, 32, 64, 30.0, 3.0, 20, 0.0),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "s%d-n%d-d%d-k%d" % c[:4])
def test_incremental_matches_full_read_and_oracle(case):
    seed, n, d, k, spread, sigma, iters, tol = case
    print("case", case, flush=True)
    X, C0 = synth.blobs(n, d, k, seed=seed, spread=spread, sigma=sigma)
    Xg, Cg = _gpu(X), _gpu(C0)
    outs, hists = [], []
    for flags in ({}, {"full_sums": True}):
        with km.KMeansMTI(Xg, Cg, **flags) as ctx:
            if not flags:
                assert ctx.path() == "lds-inc"
            for _ in range(iters):
                ctx.iterate()
            a, c = ctx.get()
            outs.append((a.cpu().numpy(), c.cpu().numpy(), ctx.centroids64()))
            hists.append(ctx.history())
    for x, y in zip(outs[0], outs[1]):
        np.testing.assert_array_equal(x, y)
    np.testing.assert_array_equal(hists[0]["changed"], hists[1]["changed"])
    assert (hists[0]["computed"] <= n * k).all()
    ref = oracle.lloyd(X, C0, iters, tol)
    a, c, st = km.run(Xg, Cg, iters, tol)
    assert st["iterations"] == ref["iters"]
    check_assign(a.cpu().numpy(), ref["assign"], ref["best"], ref["second"], "final assignment")
    check_centroids(c.cpu().numpy(), ref["C"], X, "final centroids")
    if tol == 0.0:
        np.testing.assert_array_equal(hists[0]["changed"], ref["changed"])


def test_incremental_skips_rows_and_blocks_on_separated_clusters():
    # well-separated clusters: after a few steps most points are kept by
    # Clause 1 and a batch's bounds skip the other centroid blocks
    X, C0 = synth.blobs(100000 + 9, 32, 100, seed=509, spread=40.0, sigma=1.0)
    with km.KMeansMTI(_gpu(X), _gpu(C0)) as ctx:
        for _ in range(12):
            ctx.iterate()
        h = ctx.history()
    n, k = X.shape[0], 100
    surv = n - h["clause1"][-1]
    print("clause1", h["clause1"].tolist(), "computed", h["computed"].tolist(), flush=True)
    assert h["clause1"][-1] > 0.3 * n
    assert h["computed"][-1] < surv * k   # some 32-centroid blocks skipped by Clause 2
    assert h["computed"][0] == n * k


def test_determinism_of_the_incremental_path():
    X, C0 = synth.blobs(40000, 32, 64, seed=510, spread=3.0, sigma=2.0)
    outs = []
    for _ in range(2):
        with km.KMeansMTI(_gpu(X), _gpu(C0)) as ctx:
            assert ctx.path() == "lds-inc"
            for _ in range(10):
                ctx.iterate()
            a, c = ctx.get()
            outs.append((a.cpu().numpy(), c.cpu().numpy(), ctx.centroids64()))
    for x, y in zip(outs[0], outs[1]):
        np.testing.assert_array_equal(x, y)


@pytest.mark.parametrize("k,flags,path", [
    (40, {}, "lds-inc"), (100, {}, "lds-inc"), (40, {"large_path": True}, "global-mfma"),
], ids=["lds-inc-k40", "lds-inc-k100", "global-k40"])
def test_split_bf16_band_resolves_close_pairs_like_the_oracle(k, flags, path):
    # Centroids 2000 + U(-50, 50) in every coordinate: |x| |c| is about 1.3e8,
    # so the split-bf16 error band of the expanded form (about 1.5e4 in
    # squared distance) is wider than the gap between the two nearest
    # centroids of most rows (rows placed near the bisector of two centroids:
    # gaps of about 1e3, well above the 1e-5 relative near-tie mask of the
    # comparison).  Such rows have several candidates and are decided on
    # their direct-form distances; a band that dropped the nearest centroid
    # would change assignments that the oracle fixes.
    rng = np.random.default_rng(1500 + k)
    d, n, T = 32, 40000 + 7, 3
    C0 = (2000.0 + rng.uniform(-50.0, 50.0, size=(k, d))).astype(np.float32)
    a = rng.integers(0, k, n)
    b = (a + rng.integers(1, k, n)) % k
    t = 0.5 + rng.uniform(-0.02, 0.02, n)
    X = C0[a] + t[:, None] * (C0[b] - C0[a]) + rng.normal(0.0, 0.5, size=(n, d))
    X = X.astype(np.float32)
    print("k", k, "path", path, flush=True)
    ref = oracle.lloyd(X, C0, T, 0.0, history=True)
    _, best, second, _ = oracle.assign(X, C0)
    xc = np.linalg.norm(X.astype(np.float64), axis=1) * np.linalg.norm(C0.astype(np.float64), axis=1).max()
    band = 2.0 * (778.0 + 6.9 * d) * 2.0 ** -24 * xc           # the split terms of the bound
    assert ((second - best) < band).mean() > 0.9               # most rows have several candidates
    with km.KMeansMTI(_gpu(X), _gpu(C0), **flags) as ctx:
        assert ctx.path() == path
        for _ in range(T):
            ctx.iterate()
        got, c = ctx.get()
        h = ctx.history()
    info = check_assign(got.cpu().numpy(), ref["assign"], ref["best"], ref["second"], "final assignment")
    check_centroids(c.cpu().numpy(), ref["C"], X, "final centroids")
    if info["mismatch"] == 0:
        np.testing.assert_array_equal(h["changed"], ref["changed"])
    a_gen, c_gen, _ = km.run(_gpu(X), _gpu(C0), T, 0.0, generic=True)
    np.testing.assert_array_equal(got.cpu().numpy(), a_gen.cpu().numpy())
    np.testing.assert_array_equal(c.cpu().numpy(), c_gen.cpu().numpy())
