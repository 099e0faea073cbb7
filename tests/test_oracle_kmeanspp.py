"""Pins of the k-means++ seeding oracle (CPU only).

k-means++ (paper section IV-C) draws the first seed uniformly and each later
seed with probability D(v)^2 / sum D(v)^2.  The pins below do not retype the
oracle's loops: they use closed forms on three points and on the unit square
(exact interval boundaries), numpy brute force for
the distances and the draw intervals, exact invariances and the degenerate
cases the method has (duplicates, k = 1, k = n).
"""
import numpy as np
import pytest

import oracle
import synth


def _d2_numpy(X, rows):
    X = X.astype(np.float64)
    return np.min(((X[:, None, :] - X[None, rows, :]) ** 2).sum(axis=2), axis=1)


def test_three_points_closed_form():
    # points 0, 1, 3 with the first seed at 0: D^2 = 0, 1, 9, so the second
    # seed is point 1 with probability 0.1 and point 2 with probability 0.9
    X = np.array([[0.0], [1.0], [3.0]], np.float32)
    assert oracle.kmeanspp(X, 2, np.array([0.2, 0.0999]))["idx"].tolist() == [0, 1]
    assert oracle.kmeanspp(X, 2, np.array([0.2, 0.1001]))["idx"].tolist() == [0, 2]
    r = oracle.kmeanspp(X, 2, np.array([0.2, 0.5]))
    np.testing.assert_array_equal(r["D2"], [0.0, 1.0, 0.0])
    # the first seed is floor(u0 * n)
    assert oracle.kmeanspp(X, 1, np.array([0.7]))["idx"].tolist() == [2]
    assert oracle.kmeanspp(X, 1, np.array([np.nextafter(1.0, 0.0)]))["idx"].tolist() == [2]


def test_draw_intervals_are_half_open():
    # unit square corners, first seed at the origin: D^2 = 0, 1, 1, 2, so the
    # second seed's intervals are [0, 1/4), [1/4, 1/2), [1/2, 1), all exact:
    # u on a boundary belongs to the interval that starts there
    X = np.array([[0, 0], [1, 0], [0, 1], [1, 1]], np.float32)
    for v, want in [(0.0, 1), (np.nextafter(0.25, 0.0), 1), (0.25, 2), (np.nextafter(0.5, 0.0), 2),
                    (0.5, 3), (np.nextafter(1.0, 0.0), 3)]:
        assert oracle.kmeanspp(X, 2, np.array([0.1, v]))["idx"].tolist() == [0, want], v


@pytest.mark.parametrize("seed,n,d,k", [(1, 40, 3, 6), (2, 25, 7, 5), (3, 60, 2, 4)])
def test_every_draw_lands_in_its_d2_interval(seed, n, d, k):
    # For each step, put u at the midpoint of row i's interval of the
    # cumulative D^2 / sum D^2 (numpy) and check the oracle draws row i.
    rng = np.random.default_rng(seed)
    X = rng.normal(size=(n, d)).astype(np.float32) * 3.0
    u = rng.random(k)
    base = oracle.kmeanspp(X, k, u)["idx"]
    for t in range(1, k):
        D2 = _d2_numpy(X, base[:t])
        p = D2 / D2.sum()
        hi = np.cumsum(p)
        lo = hi - p
        for i in np.nonzero(p > 1e-6)[0]:
            uu = u.copy()
            uu[t] = 0.5 * (lo[i] + hi[i])
            got = oracle.kmeanspp(X, t + 1, uu[: t + 1])["idx"]
            np.testing.assert_array_equal(got[:t], base[:t])
            assert got[t] == i, (t, i, got[t])


def test_draw_follows_d2_after_the_maximum_collapses():
    # Ten points on a line with spacing 1e-5 and one point at 1e6.  Seed 0 is
    # the first point; seed 1 is the far point (its D^2 ~ 1e12 dominates).
    # After that the maximum of D^2 falls by about 2^60, to 8.1e-9.  The draw
    # of seed 2 must still follow D^2 / sum D^2 among the near points: a
    # weight scale taken from an earlier, larger maximum would round every
    # weight to zero here.
    X = np.zeros((11, 1), np.float32)
    X[:10, 0] = (np.arange(10) * 1e-5).astype(np.float32)
    X[10, 0] = 1e6
    assert oracle.kmeanspp(X, 2, np.array([0.0, 0.5]))["idx"].tolist() == [0, 10]
    D2 = _d2_numpy(X, [0, 10])
    p = D2 / D2.sum()
    hi = np.cumsum(p)
    lo = hi - p
    for i in range(1, 10):
        u = np.array([0.0, 0.5, 0.5 * (lo[i] + hi[i])])
        assert oracle.kmeanspp(X, 3, u)["idx"].tolist() == [0, 10, i], i


def test_draw_frequencies_follow_d2():
    # many seeded draws of the second seed: chi-square against D^2 / sum D^2
    rng = np.random.default_rng(4)
    X = rng.normal(size=(12, 2)).astype(np.float32)
    draws = 20000
    counts = np.zeros(12, np.int64)
    for v in rng.random(draws):
        counts[oracle.kmeanspp(X, 2, np.array([0.0, v]))["idx"][1]] += 1
    p = _d2_numpy(X, [0])
    p = p / p.sum()
    assert counts[0] == 0
    nz = p > 0
    chi2 = (((counts - draws * p) ** 2)[nz] / (draws * p[nz])).sum()
    assert chi2 < 40.0   # 10 degrees of freedom: p-value far below 1e-4 above this


@pytest.mark.parametrize("seed,n,d,k", [(5, 3000, 16, 10), (6, 1000, 64, 30), (7, 5000, 3, 50)])
def test_d2_is_the_distance_to_the_nearest_seed(seed, n, d, k):
    X, _ = synth.blobs(n, d, k, seed=seed, spread=4.0, sigma=1.0)
    u = np.random.default_rng(seed).random(k)
    r = oracle.kmeanspp(X, k, u)
    assert len(set(r["idx"].tolist())) == k   # distinct rows: a drawn row has weight 0
    np.testing.assert_allclose(r["D2"], _d2_numpy(X, r["idx"]), rtol=1e-12, atol=0)
    np.testing.assert_array_equal(r["C"], X[r["idx"]])
    assert (r["D2"][r["idx"]] == 0).all()


def test_prefix_property():
    # the first t seeds do not depend on k
    X, _ = synth.blobs(2000, 8, 9, seed=8)
    u = np.random.default_rng(8).random(9)
    a = oracle.kmeanspp(X, 9, u)["idx"]
    b = oracle.kmeanspp(X, 5, u[:5])["idx"]
    np.testing.assert_array_equal(a[:5], b)


def test_power_of_two_scale_gives_the_same_seeds():
    # D^2 scales by 4^e exactly and the weight scale follows, so the integer
    # weights and hence the draws are identical
    X, _ = synth.blobs(3000, 5, 12, seed=9, spread=3.0)
    u = np.random.default_rng(9).random(12)
    a = oracle.kmeanspp(X, 12, u)
    for e in (-7, 3, 11):
        b = oracle.kmeanspp((X.astype(np.float64) * 2.0 ** e).astype(np.float32), 12, u)
        np.testing.assert_array_equal(a["idx"], b["idx"])
        np.testing.assert_array_equal(a["D2"] * 4.0 ** e, b["D2"])


def test_duplicates_and_exhausted_weights():
    # three distinct points, each repeated: the first three seeds are one copy
    # of each; the fourth draw has W = 0 and falls back to the uniform rule
    base = np.array([[0.0, 0.0], [5.0, 1.0], [-2.0, 7.0]], np.float32)
    X = np.repeat(base, [4, 3, 5], axis=0)
    rng = np.random.default_rng(10)
    for _ in range(20):
        u = rng.random(4)
        r = oracle.kmeanspp(X, 4, u)
        groups = {tuple(X[i]) for i in r["idx"][:3]}
        assert len(groups) == 3
        assert r["idx"][3] == min(int(u[3] * len(X)), len(X) - 1)
        assert (r["D2"] == 0).all()


def test_k_equals_n_draws_every_row_once():
    rng = np.random.default_rng(11)
    X = rng.normal(size=(30, 4)).astype(np.float32)
    r = oracle.kmeanspp(X, 30, rng.random(30))
    assert sorted(r["idx"].tolist()) == list(range(30))
    assert (r["D2"] == 0).all()


def test_bad_arguments_are_refused():
    X = np.zeros((5, 2), np.float32)
    with pytest.raises(ValueError):
        oracle.kmeanspp(X, 2, np.array([0.5, 1.0]))
    with pytest.raises(ValueError):
        oracle.kmeanspp(X, 6, np.full(6, 0.5))
    with pytest.raises(ValueError):
        oracle.kmeanspp(X, 2, np.array([-0.1, 0.5]))
