"""Pins of the spherical k-means oracle (CPU only).

Spherical k-means (the paper's section on sk-means among the applications)
projects the points to the unit sphere and uses the cosine for proximity;
the update reading is the members' unit-vector sum projected to the sphere.
The pins below do not retype the oracle's loops: they use numpy matrix forms,
closed forms on symmetric data, exact invariances and the monotone
objective.
"""
import numpy as np
import pytest

import oracle
import synth


def _unit(A):
    A = np.asarray(A, np.float64)
    r = np.linalg.norm(A, axis=1, keepdims=True)
    return np.where(r > 0, A / np.where(r > 0, r, 1.0), 0.0)


@pytest.mark.parametrize("seed,n,d,k", [(1, 500, 3, 4), (2, 800, 16, 7), (3, 300, 40, 12)])
def test_one_step_is_cosine_argmax_then_projected_sum(seed, n, d, k):
    X, C0 = synth.blobs(n, d, k, seed=seed, spread=2.0, sigma=1.0)
    r = oracle.spherical(X, C0, 1)
    cos = _unit(X) @ _unit(C0).T                     # every cosine at once
    np.testing.assert_array_equal(r["assign"], np.argmax(cos, axis=1))
    S = np.zeros((k, d))
    np.add.at(S, r["assign"], _unit(X))
    np.testing.assert_allclose(r["C"], _unit(S), rtol=0, atol=1e-13)
    srt = np.sort(2.0 - 2.0 * cos, axis=1)
    np.testing.assert_allclose(r["best"], srt[:, 0], rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["second"], srt[:, 1], rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed,n,d,k", [(4, 2000, 8, 5), (5, 3000, 16, 10), (6, 1500, 32, 20)])
def test_objective_never_increases(seed, n, d, k):
    # sum of squared chord distances = 2n - 2 sum cos: the projected mean
    # maximises each cluster's cosine sum and the argmax never lowers it.
    X, C0 = synth.blobs(n, d, k, seed=seed, spread=3.0, sigma=2.0)
    r = oracle.spherical(X, C0, 30)
    J = r["objective"]
    assert np.all(np.diff(J) <= 1e-9 * J[0])
    assert np.linalg.norm(r["C"], axis=1) == pytest.approx(np.ones(k), abs=1e-15)


def test_power_of_two_scaling_is_invisible():
    # x * 2^e has the same unit vector bit for bit, so the whole run is equal.
    X, C0 = synth.blobs(1200, 10, 6, seed=7, spread=2.0)
    rng = np.random.default_rng(7)
    e = rng.integers(-20, 20, size=(X.shape[0], 1)).astype(np.float64)
    Xs = (X.astype(np.float64) * 2.0 ** e).astype(np.float32)
    C0s = (C0.astype(np.float64) * 2.0 ** rng.integers(-5, 5, size=(6, 1))).astype(np.float32)
    a = oracle.spherical(X, C0, 15)
    b = oracle.spherical(Xs, C0s, 15)
    np.testing.assert_array_equal(a["assign"], b["assign"])
    np.testing.assert_array_equal(a["C"], b["C"])
    assert a["iters"] == b["iters"]


def test_symmetric_pairs_converge_to_the_axes():
    # Two mirror pairs (p, q) and (p, -q) around each axis: each cluster's
    # unit sum lies exactly on its axis, so the centroids are e1 and e2.
    pts = []
    for p, q in [(3.0, 1.0), (5.0, 0.5), (2.0, 0.25)]:
        pts += [(p, q), (p, -q), (q, p), (-q, p)]
    X = np.array(pts, np.float32)
    r = oracle.spherical(X, X[[0, 2]], 10)
    np.testing.assert_array_equal(r["C"], np.array([[1.0, 0.0], [0.0, 1.0]]))
    np.testing.assert_array_equal(r["assign"], np.array([0, 0, 1, 1] * 3))


def test_k1_centroid_is_the_projected_sum_of_all_unit_vectors():
    X, C0 = synth.blobs(999, 6, 1, seed=8, spread=1.0)
    r = oracle.spherical(X, C0, 3)
    want = _unit(_unit(X).sum(axis=0, keepdims=True))[0]
    np.testing.assert_allclose(r["C"][0], want, rtol=0, atol=1e-14)
    assert (r["assign"] == 0).all()


def test_zero_rows_tie_everywhere_and_zero_centroids_are_refused():
    X, C0 = synth.blobs(200, 4, 3, seed=9, spread=2.0)
    X = X.copy()
    X[[5, 17]] = 0.0                                   # no direction: cosine 0 with every centroid
    r = oracle.spherical(X, C0, 1)
    assert r["assign"][5] == 0 and r["assign"][17] == 0   # all tie: lowest index
    C0z = C0.copy()
    C0z[1] = 0.0
    with pytest.raises(ValueError):
        oracle.spherical(X, C0z, 1)
