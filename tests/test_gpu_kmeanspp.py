"""k-means++ seeding on the GPU (kmeans_pp_seed through the C ABI) against
the float64 seeding oracle.

Seeding is index work decided by float64 arithmetic that both sides carry out
in the same order, so the bar is bit-exact: identical seed indices, seed rows
and D2 values, with and without the triangle-inequality skip.  The full-size
workloads are checked whole where the oracle finishes in seconds, else on the
prefix of the draws (the first t seeds do not depend on k) and on sampled
rows.
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


def _check(got, ref, X):
    idx = got["idx"].cpu().numpy()
    np.testing.assert_array_equal(idx, ref["idx"])
    np.testing.assert_array_equal(got["C"].cpu().numpy(), X[ref["idx"]])
    np.testing.assert_array_equal(got["D2"].cpu().numpy(), ref["D2"])


CASES = [
    # seed, n, d, k
    (301, 3000 + 5, 16, 10),
    (302, 5000 + 3, 3, 20),
    (303, 20000 + 17, 64, 50),
    (304, 8000 + 1, 100, 40),     # wide rows: seed-to-seed table by whole waves
    (305, 2 * 2048 + 1, 5, 3),    # one row past two chunks
    (306, 2048, 16, 64),          # exactly one chunk
    (307, 50000 + 11, 32, 128),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "s%d-n%d-d%d-k%d" % c)
@pytest.mark.parametrize("prune", [True, False], ids=["prune", "noprune"])
def test_seeding_is_bit_exact(case, prune):
    seed, n, d, k = case
    print("case", case, prune, flush=True)
    X, _ = synth.blobs(n, d, max(k // 2, 1), seed=seed, spread=4.0, sigma=1.0)
    u = np.random.default_rng(seed).random(k)
    ref = oracle.kmeanspp(X, k, u)
    got = km.kmeanspp(_gpu(X), k, u, prune=prune, count=True)
    _check(got, ref, X)
    st = got["stats"]
    assert 0 < st["computed"] <= n * k and st["passes"] == k
    assert 0 <= st["improved"] <= st["computed"] - n
    if not prune:
        assert st["computed"] == n * k


def test_pruning_skips_distances_on_clustered_data():
    X, _ = synth.blobs(100000 + 7, 16, 50, seed=308, spread=20.0, sigma=1.0)
    u = np.random.default_rng(308).random(50)
    ref = oracle.kmeanspp(X, 50, u)
    got = km.kmeanspp(_gpu(X), 50, u, timing=True)
    _check(got, ref, X)
    st = got["stats"]
    assert st["computed"] < 0.7 * X.shape[0] * 50, st
    assert st["pass_ms"] > st["later_pass_ms"] > 0 and st["draw_ms"] > 0


def test_degenerate_cases():
    # n = 1; k = n; every row drawn once; duplicates exhaust the weights
    # (W = 0 draws uniformly); exact interval boundaries on the unit square
    X = np.array([[1.0, 2.0, 3.0, 4.0]], np.float32)
    _check(km.kmeanspp(_gpu(X), 1, [0.3]), oracle.kmeanspp(X, 1, np.array([0.3])), X)
    rng = np.random.default_rng(309)
    X = rng.normal(size=(33, 6)).astype(np.float32)
    u = rng.random(33)
    ref = oracle.kmeanspp(X, 33, u)
    assert sorted(ref["idx"].tolist()) == list(range(33))
    _check(km.kmeanspp(_gpu(X), 33, u), ref, X)
    base = np.array([[0.0, 0.0], [5.0, 1.0], [-2.0, 7.0]], np.float32)
    X = np.repeat(base, [700, 900, 2000], axis=0)
    for _ in range(5):
        u = rng.random(6)
        ref = oracle.kmeanspp(X, 6, u)
        _check(km.kmeanspp(_gpu(X), 6, u), ref, X)
        _check(km.kmeanspp(_gpu(X), 6, u, prune=False), ref, X)
    X = np.array([[0, 0], [1, 0], [0, 1], [1, 1]], np.float32)
    for v in [0.0, np.nextafter(0.25, 0.0), 0.25, np.nextafter(0.5, 0.0), 0.5, np.nextafter(1.0, 0.0)]:
        u = np.array([0.1, v])
        _check(km.kmeanspp(_gpu(X), 2, u), oracle.kmeanspp(X, 2, u), X)


def test_workspace_reuse_and_errors():
    X, _ = synth.blobs(6000, 8, 5, seed=310)
    Xg = _gpu(X)
    ws = torch.empty(km.kmeanspp_workspace_bytes(6000, 8, 12) + 256, dtype=torch.uint8, device=DEV)
    rng = np.random.default_rng(310)
    for k in (12, 4, 12):   # stale contents of an earlier call must not matter
        u = rng.random(k)
        _check(km.kmeanspp(Xg, k, u, workspace=ws), oracle.kmeanspp(X, k, u), X)
    with pytest.raises(N.KMError):
        km.kmeanspp(Xg, 3, [0.5, 1.0, 0.5])
    with pytest.raises(ValueError):
        km.kmeanspp(Xg, 12, rng.random(12), workspace=ws[:1000])


@pytest.mark.parametrize("name", ["aniso-8M-d16-k10"])
def test_full_size_workload_is_bit_exact(name):
    X, _, w = synth.make(name)
    u = np.random.default_rng(311).random(w.k)
    print("workload", name, flush=True)
    ref = oracle.kmeanspp(X, w.k, u)
    _check(km.kmeanspp(_gpu(X), w.k, u), ref, X)


def test_large_k_workload_prefix_and_sampled_rows():
    # 2M x 256, k = 1000: the first 12 draws against the oracle (prefix
    # property), then every row's D2 on a sample against a float64 brute
    # force over all 1000 seeds
    X, _, w = synth.make("blobs-2M-d256-k1000")
    u = np.random.default_rng(312).random(w.k)
    print("workload", w.name, flush=True)
    got = km.kmeanspp(_gpu(X), w.k, u, count=True)
    idx = got["idx"].cpu().numpy()
    ref = oracle.kmeanspp(X, 12, u[:12])
    np.testing.assert_array_equal(idx[:12], ref["idx"])
    assert len(set(idx.tolist())) == w.k
    np.testing.assert_array_equal(got["C"].cpu().numpy(), X[idx])
    rows = np.random.default_rng(313).choice(X.shape[0], 1500, replace=False)
    S = X[idx].astype(np.float64)
    xs = X[rows].astype(np.float64)
    bf = ((xs * xs).sum(1)[:, None] - 2.0 * xs @ S.T + (S * S).sum(1)[None, :]).min(axis=1)
    D2 = got["D2"].cpu().numpy()[rows]
    np.testing.assert_allclose(D2, np.maximum(bf, 0.0), rtol=1e-9, atol=1e-9 * float(bf.max()))
    assert got["stats"]["computed"] < X.shape[0] * w.k


def test_best_of_restarts_matches_the_oracle():
    # The paper's k-means++ with r restarts: seed, run, keep the least final
    # inertia.  Each run against the oracle's seeding and Lloyd's run.
    X, _ = synth.blobs(20000 + 13, 16, 12, seed=314, spread=3.0, sigma=1.5)
    k, r, iters = 12, 4, 15
    U = np.random.default_rng(314).random((r, k))
    got = km.run_pp_best(_gpu(X), k, U, iters)
    inert = []
    for i in range(r):
        seeds = oracle.kmeanspp(X, k, U[i])
        ref = oracle.lloyd(X, seeds["C"], iters)
        inert.append(ref["inertia"][-1])
        assert got["inertia"][i] == pytest.approx(inert[-1], rel=1e-5)
    want = int(np.argmin(inert))
    srt = np.sort(inert)
    if srt[1] - srt[0] > 1e-4 * srt[0]:   # a clear winner
        assert got["best"] == want
    ref = oracle.lloyd(X, oracle.kmeanspp(X, k, U[got["best"]])["C"], iters)
    check_assign(got["assign"].cpu().numpy(), ref["assign"], ref["best"], ref["second"], "best run")
    check_centroids(got["C"].cpu().numpy(), ref["C"], X, "best run")
