"""The one-launch streaming step (d = 16, k <= 16) against the oracle and
against the general kernels (KM_FLAG_GENERIC), through the C ABI.

Sizes span one partial tile, several tiles per block, and enough blocks for
several completion groups (the group and final reductions of the last
blocks); every case has a ragged last tile.
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
    # seed, n, k, spread, sigma, iters, tol
    (101, 1, 1, 3.0, 1.0, 3, 0.0),
    (102, 37, 5, 3.0, 1.0, 10, 0.0),
    (103, 255, 16, 2.0, 1.0, 15, 0.0),
    (104, 3 * 256 + 1, 2, 1.0, 1.0, 20, 0.0),
    (105, 20000 + 13, 10, 3.0, 2.0, 30, 0.0),
    (106, 50000 + 77, 16, 1.5, 1.5, 30, 0.001),
    (107, 400000 + 5, 10, 4.0, 2.0, 12, 0.0),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "s%d-n%d-k%d" % c[:3])
@pytest.mark.parametrize("stats", [False, True], ids=["incremental", "full+inertia"])
def test_stream_matches_oracle(case, stats):
    seed, n, k, spread, sigma, iters, tol = case
    print("case", case, stats, flush=True)
    X, C0 = synth.blobs(n, 16, k, seed=seed, spread=spread, sigma=sigma)
    ref = oracle.lloyd(X, C0, iters, tol)
    a, c, st = km.run(_gpu(X), _gpu(C0), iters, tol, stats=stats)
    assert st["iterations"] == ref["iters"]
    check_assign(a.cpu().numpy(), ref["assign"], ref["best"], ref["second"], "final assignment")
    check_centroids(c.cpu().numpy(), ref["C"], X, "final centroids")
    if stats:
        assert st["inertia_last"] == pytest.approx(ref["inertia"][-1], rel=1e-5)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "s%d-n%d-k%d" % c[:3])
@pytest.mark.parametrize("prune", [True, False], ids=["prune", "noprune"])
def test_stream_paths_are_bitwise_identical_to_generic_path(case, prune):
    # incremental sums (default), full sums every step, full sums with inertia,
    # and the general kernels: same assignments, centroids and changed counts
    seed, n, k, spread, sigma, iters, tol = case
    print("case", case, prune, flush=True)
    X, C0 = synth.blobs(n, 16, k, seed=seed, spread=spread, sigma=sigma)
    Xg, Cg = _gpu(X), _gpu(C0)
    modes = [dict(), dict(full_sums=True), dict(stats=True), dict(stats=True, generic=True)]
    paths, hists, outs = [], [], []
    for m in modes:
        with km.KMeansMTI(Xg, Cg, prune=prune, **m) as ctx:
            for _ in range(iters):
                ctx.iterate()
            a, c = ctx.get()
            outs.append((a.cpu().numpy(), c.cpu().numpy(), ctx.centroids64()))
            hists.append(ctx.history())
            paths.append(ctx.path())
    assert paths == ["stream-d16", "stream-d16-full", "stream-d16-full", "lds-vector"]
    for o, h in zip(outs[1:], hists[1:]):
        np.testing.assert_array_equal(outs[0][0], o[0])
        np.testing.assert_array_equal(outs[0][1], o[1])
        np.testing.assert_array_equal(outs[0][2], o[2])
        np.testing.assert_array_equal(hists[0]["changed"], h["changed"])
    # The inertia sums each point's float32 distance; a near tie decided again
    # in float64 contributes that distance rounded to float32.  The paths
    # form their candidate sets differently (certified expanded-form
    # candidates on the streaming path), so a few near-tie points can take the
    # float64 decision on one path only: a difference of a few float32 units
    # of one term.
    np.testing.assert_allclose(hists[2]["inertia"], hists[3]["inertia"], rtol=1e-9)
    if not prune:
        assert (hists[0]["computed"] == n * k).all()


def test_first_step_exact_ties_take_the_lowest_index():
    # Every other row lies on the bisector of c0 and c1 (their only difference
    # is the sign of coordinate 0, which is 0 in those rows): exact ties in
    # float32 and float64.  The matrix-core first step finds both centroids
    # inside its candidate band, decides those rows on their direct-form
    # distances and in float64, and must give the oracle's lowest index; the
    # rows are spread over many 64-point tiles with a ragged end.
    rng = np.random.default_rng(120)
    n, k = 9000 + 21, 7
    C0 = rng.uniform(-30.0, 30.0, size=(k, 16)).astype(np.float32)
    C0[1] = C0[0]
    C0[0, 0], C0[1, 0] = 2.0, -2.0
    X = (C0[rng.integers(0, k, n)] + rng.integers(-3, 4, size=(n, 16))).astype(np.float32)
    X[::2] = C0[0] + rng.integers(-3, 4, size=(len(X[::2]), 16)).astype(np.float32)
    X[::2, 0] = 0.0
    ref = oracle.lloyd(X, C0, 1, 0.0)
    tied = (X[:, 0] == 0.0) & (ref["assign"] == 0)
    assert tied.sum() > n // 4
    with km.KMeansMTI(_gpu(X), _gpu(C0)) as ctx:
        assert ctx.path() == "stream-d16"
        ctx.iterate()
        a, _ = ctx.get(centroids=False)
        np.testing.assert_array_equal(a.cpu().numpy(), ref["assign"])
        np.testing.assert_allclose(ctx.centroids64(), ref["C"], rtol=1e-12, atol=1e-12)
        assert ctx.history()["rechecks"][0] >= tied.sum()


def test_incremental_trajectory_every_step_matches_oracle():
    X, C0 = synth.blobs(70000 + 9, 16, 12, seed=112, spread=3.0, sigma=1.5)
    T = 15
    ref = oracle.lloyd(X, C0, T, history=True)
    with km.KMeansMTI(_gpu(X), _gpu(C0)) as ctx:
        assert ctx.path() == "stream-d16"
        for t in range(T):
            ch = ctx.iterate(sync=True)
            a, c = ctx.get()
            prev = None if t == 0 else ref["assign_hist"][t - 1]
            _, b, s, _ = oracle.assign(X, ref["C_hist"][t], prev=prev)
            info = check_assign(a.cpu().numpy(), ref["assign_hist"][t], b, s, "step %d" % t)
            if info["mismatch"] == 0:
                assert ch == ref["changed"][t]
            np.testing.assert_allclose(ctx.centroids64(), ref["C_hist"][t + 1], rtol=1e-9, atol=1e-9)
        h = ctx.history()
    np.testing.assert_array_equal(h["changed"], ref["changed"])
    assert np.isnan(h["inertia"]).all()


def test_stream_trajectory_and_history():
    X, C0 = synth.blobs(60000 + 3, 16, 10, seed=111, spread=3.0, sigma=2.0)
    T = 12
    ref = oracle.lloyd(X, C0, T, history=True)
    with km.KMeansMTI(_gpu(X), _gpu(C0), stats=True, timing=True) as ctx:
        for t in range(T):
            ch = ctx.iterate(sync=True)
            a, c = ctx.get()
            prev = None if t == 0 else ref["assign_hist"][t - 1]
            _, b, s, _ = oracle.assign(X, ref["C_hist"][t], prev=prev)
            info = check_assign(a.cpu().numpy(), ref["assign_hist"][t], b, s, "step %d" % t)
            if info["mismatch"] == 0:
                assert ch == ref["changed"][t]
            check_centroids(c.cpu().numpy(), ref["C_hist"][t + 1], X, "step %d" % t)
            np.testing.assert_allclose(ctx.centroids64(), ref["C_hist"][t + 1], rtol=1e-9, atol=1e-9)
        h = ctx.history()
        tm = ctx.timing()
    np.testing.assert_array_equal(h["changed"], ref["changed"])
    np.testing.assert_allclose(h["inertia"], ref["inertia"], rtol=1e-5)
    assert (h["computed"] <= X.shape[0] * 10).all() and h["clause1"][0] == 0
    assert tm["iters"] == T and tm["assign_ms"] > 0
    # two launches per step (streaming kernel, finishing block in the update
    # slot): the reduce and table intervals enclose no kernel
    assert tm["update_ms"] > 0 and tm["reduce_ms"] + tm["table_ms"] < 0.02 * T


def test_stream_repeated_runs_reuse_accumulation_rows():
    # Many steps per context, two contexts: the accumulation rows must be
    # back at zero after every step, or a later step would double count.
    X, C0 = synth.blobs(300000 + 11, 16, 8, seed=121, spread=3.0, sigma=1.5)
    ref = oracle.lloyd(X, C0, 40, 0.0)
    Xg, Cg = _gpu(X), _gpu(C0)
    for _ in range(2):
        a, c, st = km.run(Xg, Cg, 40, 0.0)
        assert st["iterations"] == ref["iters"]
        check_assign(a.cpu().numpy(), ref["assign"], ref["best"], ref["second"], "final assignment")
        check_centroids(c.cpu().numpy(), ref["C"], X, "final centroids")


@pytest.mark.parametrize("d,k,flags,path", [
    (16, 10, {}, "stream-d16"), (16, 16, {}, "stream-d16"), (16, 10, {"full_sums": True}, "stream-d16-full"),
    (16, 10, {"stats": True}, "stream-d16-full"), (16, 10, {"generic": True}, "lds-vector"),
    (16, 17, {}, "lds-inc"), (32, 10, {}, "lds-inc"), (32, 100, {}, "lds-inc"),
    (16, 17, {"full_sums": True}, "lds-mfma"), (32, 10, {"full_sums": True}, "lds-vector"),
    (32, 100, {"vector_only": True}, "lds-vector"), (16, 10, {"large_path": True}, "global-mfma"),
])
def test_path_selection(d, k, flags, path):
    X, C0 = synth.blobs(1000, d, k, seed=131)
    with km.KMeansMTI(_gpu(X), _gpu(C0), **flags) as ctx:
        assert ctx.path() == path


# Sizes at the incremental kernel's tiling edges: 1024-point wave tiles, eight
# waves per block, blocks owning fewer tiles than waves, one tile short of or
# past a whole number of blocks' tiles, and a ragged last sub-tile.
EDGE_N = [1023, 1024, 1025, 8 * 1024 - 1, 8 * 1024, 8 * 1024 + 1, 16 * 1024 + 3, 300 * 1024 + 257]


@pytest.mark.parametrize("n", EDGE_N)
def test_incremental_tiling_edges_match_oracle_and_generic_path(n):
    rng = np.random.default_rng(9000 + n)
    k = int(rng.integers(1, 17))
    print("n", n, "k", k, flush=True)
    X, C0 = synth.blobs(n, 16, k, seed=9000 + n, spread=3.0, sigma=1.5)
    iters = 12
    ref = oracle.lloyd(X, C0, iters, 0.0)
    Xg, Cg = _gpu(X), _gpu(C0)
    with km.KMeansMTI(Xg, Cg) as ctx:
        assert ctx.path() == "stream-d16"
    a, c, st = km.run(Xg, Cg, iters, 0.0, stats=False)
    assert st["iterations"] == ref["iters"]
    check_assign(a.cpu().numpy(), ref["assign"], ref["best"], ref["second"], "final assignment")
    check_centroids(c.cpu().numpy(), ref["C"], X, "final centroids")
    a2, c2, _ = km.run(Xg, Cg, iters, 0.0, generic=True)
    assert torch.equal(a, a2) and torch.equal(c, c2)


def test_dense_step_settles_listed_ties_like_the_oracle():
    # Two fixed centroids (-2, 0, ...) and (2, 0, ...): every cluster's mean is
    # its initial centroid (rows in +-offset pairs; each tie row x0 = 0 has a
    # partner at x0 = -4), so the drift is zero and the tie rows (x0 = 0,
    # equidistant in float32 and float64) survive Clause 1 in every step with
    # two candidates.  In the streamed first incremental step they are listed
    # and settled as gathered survivors; 44 % of the rows are ties over about
    # seven 64-row tiles per wave, so each wave's list fills and is drained
    # in the middle of its tiles.  The
    # oracle's lowest index and the incumbent rule both give cluster 0.
    rng = np.random.default_rng(140)
    m = 200000
    y = rng.integers(-3, 4, size=(2 * m, 15))
    y[:, 0] = np.where(y[:, 0] == 0, 1, y[:, 0])                 # |y| > 0: a bound above s(c0) = 2
    ties = np.concatenate([np.zeros((2 * m, 1)), np.concatenate([y[:m], -y[:m]])], axis=1)
    comp = np.concatenate([np.full((2 * m, 1), -4.0), np.concatenate([y[m:], -y[m:]])], axis=1)
    off = rng.integers(-1, 2, size=(m // 8, 16))
    base0 = np.concatenate([off, -off]) + np.eye(16)[0] * -2.0
    off = rng.integers(-1, 2, size=(m // 8, 16))
    base1 = np.concatenate([off, -off]) + np.eye(16)[0] * 2.0
    X = np.concatenate([ties, comp, base0, base1]).astype(np.float32)
    X = X[rng.permutation(len(X))]
    C0 = np.zeros((2, 16), np.float32)
    C0[0, 0], C0[1, 0] = -2.0, 2.0
    n, T = len(X), 3
    print("n", n, "ties", 2 * m, flush=True)
    ref = oracle.lloyd(X, C0, T, 0.0)
    assert (ref["assign"][X[:, 0] == 0.0] == 0).all()
    outs = []
    for flags in ({}, {"full_sums": True}):
        with km.KMeansMTI(_gpu(X), _gpu(C0), **flags) as ctx:
            for _ in range(T):
                ctx.iterate()
            a, _ = ctx.get(centroids=False)
            outs.append((a.cpu().numpy(), ctx.centroids64(), ctx.history()))
    a, c64, h = outs[0]
    np.testing.assert_array_equal(a, ref["assign"])
    np.testing.assert_allclose(c64, ref["C"], rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(h["changed"], [n, 0, 0])
    assert (h["rechecks"][1:] >= 2 * m).all()                    # every tie row decided in float64
    np.testing.assert_array_equal(a, outs[1][0])
    np.testing.assert_array_equal(c64, outs[1][1])


def _sample_rows(n, d):
    # The fixed sample of X the set-up reads: 16 chunks, chunk c from row
    # c * n // 16, max(1, 1024 // d) rows, cut at n.
    rows = max(1, 1024 // d)
    out = np.zeros(n, bool)
    for c in range(16):
        r0 = c * n // 16
        out[r0:min(r0 + rows, n)] = True
    return out


@pytest.mark.parametrize("big", [3.0e3, 1.0e15], ids=["x3e3", "x1e15"])
def test_first_step_corrects_its_sums_when_x_exceeds_the_sample_bound(big):
    # The stream path's first step forms its sums at the scale of a bound 16
    # times the largest |x| of the sample and finds the largest |x| itself; a
    # row outside the sample beyond that bound makes it correct its sums to
    # the final scale (for 1e15 the first images are not even exact integers).
    # The results must be bitwise those of the same path after a full set-up
    # scan (validate) and of the general kernels, and the oracle's for the
    # moderate outlier.
    n, k = 100_000 + 11, 8
    X, C0 = synth.blobs(n, 16, k, seed=4242, spread=3.0, sigma=1.0)
    samp = _sample_rows(n, 16)
    out = np.flatnonzero(~samp)
    r = int(out[len(out) // 2])
    X = X.copy()
    X[r, 3] = big
    assert np.frexp(np.float32(big))[1] > np.frexp(np.abs(X[samp]).max())[1] + 4   # past the bound
    print("outlier row", r, big, flush=True)
    iters = 8
    Xg, Cg = _gpu(X), _gpu(C0)
    with km.KMeansMTI(Xg, Cg) as ctx:
        assert ctx.path() == "stream-d16"
    a, c, st = km.run(Xg, Cg, iters, 0.0)
    a1, c1, st1 = km.run(Xg, Cg, iters, 0.0, validate=True)
    a2, c2, _ = km.run(Xg, Cg, iters, 0.0, generic=True)
    assert torch.equal(a, a1) and torch.equal(c, c1) and st["iterations"] == st1["iterations"]
    assert torch.equal(a, a2) and torch.equal(c, c2)
    if big < 1e6:
        ref = oracle.lloyd(X, C0, iters, 0.0)
        assert st["iterations"] == ref["iters"]
        check_assign(a.cpu().numpy(), ref["assign"], ref["best"], ref["second"], "final assignment")
        check_centroids(c.cpu().numpy(), ref["C"], X, "final centroids")
