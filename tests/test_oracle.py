"""Pins for the CPU oracle (plain float64 Lloyd's) and the CPU MTI reference.

Every check here ties the oracle to something other than itself: values
derived by hand from the definitions (tests/golden), exact rational
arithmetic, closed forms, independent libraries (scipy's vector quantiser,
scikit-learn's Lloyd k-means), exhaustive enumeration on tiny inputs, and the
mathematical invariants of Lloyd's algorithm.  The MTI reference is pinned by
the property the paper's method rests on: pruning never changes an
assignment (section III-C).
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# --------------------------------------------------------------------------- golden


def test_worked_example_steps():
    g = _load("worked_2d.json")
    X = np.array(g["X"], np.float32)
    C0 = np.array(g["C0"], np.float64)
    r = oracle.lloyd(X, C0, max_iters=3, tol=0.0, history=True)
    assert r["iters"] == 3
    for t, st in enumerate(g["steps"]):
        assert r["assign_hist"][t].tolist() == st["assign"]
        assert int(r["changed"][t]) == st["changed"]
        assert r["inertia"][t] == pytest.approx(st["inertia"], rel=1e-15, abs=0)
        np.testing.assert_allclose(r["C_hist"][t + 1], np.array(st["C_after"]), rtol=1e-15, atol=0)


@pytest.mark.parametrize("run", _load("worked_2d.json")["runs"])
def test_worked_example_stopping(run):
    g = _load("worked_2d.json")
    X = np.array(g["X"], np.float32)
    r = oracle.lloyd(X, np.array(g["C0"], np.float64), run["max_iters"], run["tol"])
    assert r["iters"] == run["iters"]
    last = g["steps"][run["iters"] - 1]
    assert r["assign"].tolist() == last["assign"]
    np.testing.assert_allclose(r["C"], np.array(last["C_after"]), rtol=1e-15, atol=0)


@pytest.mark.parametrize("case", _load("ties_1d.json")["cases"], ids=lambda c: c["name"])
def test_tie_and_empty_rules(case):
    X = np.array(case["X"], np.float32)
    C0 = np.array(case["C0"], np.float64)
    r = oracle.lloyd(X, C0, case["max_iters"], 0.0, history=True)
    assert r["assign_hist"].tolist() == case["assign_hist"]
    np.testing.assert_array_equal(r["C"], np.array(case["C"]))
    m = oracle.mti(X, C0, case["max_iters"], 0.0, history=True)
    assert m["assign_hist"].tolist() == case["assign_hist"]


# --------------------------------------------------------------------------- exact arithmetic


def test_update_is_exact_mean_on_dyadic_data():
    rng = np.random.default_rng(7)
    n, d, k = 64, 5, 4
    X = (rng.integers(-40, 40, size=(n, d)) / 4.0).astype(np.float32)
    a = rng.integers(0, k, size=n).astype(np.int32)
    Cold = rng.normal(size=(k, d))
    Cn, cnt = oracle.update(X, a, Cold)
    assert cnt.sum() == n
    for j in range(k):
        members = [i for i in range(n) if a[i] == j]
        assert cnt[j] == len(members)
        for m in range(d):
            if members:
                exact = sum(Fraction(float(X[i, m])) for i in members) / len(members)
                assert Cn[j, m] == float(exact)      # correctly rounded mean
            else:
                assert Cn[j, m] == Cold[j, m]


def test_assign_step_matches_exact_rational_argmin():
    rng = np.random.default_rng(11)
    n, d, k = 40, 3, 5
    X = (rng.integers(-20, 20, size=(n, d)) / 2.0).astype(np.float32)
    Cm = rng.integers(-20, 20, size=(k, d)) / 2.0
    a, best, second, changed = oracle.assign(X, Cm)
    assert changed == n
    for i in range(n):
        D = [sum((Fraction(float(X[i, m])) - Fraction(float(Cm[j, m]))) ** 2 for m in range(d))
             for j in range(k)]
        lo = min(D)
        assert a[i] == D.index(lo)                   # lowest index among exact ties
        assert best[i] == float(lo)
        rest = sorted(D)[1]
        assert second[i] == float(rest)


# --------------------------------------------------------------------------- closed forms / invariants


def test_k1_is_global_mean():
    X, _ = synth.blobs(500, 7, 1, seed=3)
    C0 = X[:1].astype(np.float64)
    r = oracle.lloyd(X, C0, max_iters=4, history=True)
    mean = np.array([math.fsum(X[:, m].astype(np.float64)) / X.shape[0] for m in range(X.shape[1])])
    np.testing.assert_allclose(r["C"], mean[None, :], rtol=1e-13, atol=1e-13)
    assert (r["assign"] == 0).all()
    assert r["changed"].tolist() == [500, 0, 0, 0]
    # after step 0 the centroid no longer moves
    np.testing.assert_array_equal(r["C_hist"][1], r["C_hist"][4])


def test_k_equals_n_distinct_points_zero_inertia():
    X, _ = synth.blobs(12, 3, 12, seed=5)
    r = oracle.lloyd(X, X.astype(np.float64), max_iters=3, history=True)
    assert r["assign"].tolist() == list(range(12))
    assert (r["inertia"] == 0).all()
    np.testing.assert_array_equal(r["C"], X.astype(np.float64))


@pytest.mark.parametrize("seed,n,d,k", [(1, 3000, 2, 6), (2, 2000, 16, 12), (3, 1500, 5, 40)])
def test_inertia_non_increasing_and_counts(seed, n, d, k):
    X, C0 = synth.blobs(n, d, k, seed=seed, spread=4.0, sigma=1.5)
    r = oracle.lloyd(X, C0, max_iters=25, history=True)
    J = r["inertia"]
    assert np.all(J[1:] <= J[:-1] * (1 + 1e-12))
    for t in range(r["iters"]):
        _, cnt = oracle.update(X, r["assign_hist"][t], r["C_hist"][t])
        assert cnt.sum() == n


def test_converged_partition_is_fixed_point():
    X, C0 = synth.blobs(800, 4, 6, seed=9)
    r = oracle.lloyd(X, C0, max_iters=100, tol=0.0)
    a2, _, _, ch = oracle.assign(X, r["C"], prev=r["assign"])
    assert ch == 0 and (a2 == r["assign"]).all()
    C2, _ = oracle.update(X, r["assign"], r["C"])
    np.testing.assert_allclose(C2, r["C"], rtol=1e-14, atol=1e-14)


def test_duplicate_points():
    X, C0 = synth.blobs(300, 3, 4, seed=12)
    X = np.concatenate([X, X[:150], X[:50]])
    r = oracle.lloyd(X, C0, max_iters=15, history=True)
    # duplicated rows always share their assignment
    assert (r["assign"][300:450] == r["assign"][:150]).all()
    assert (r["assign"][450:] == r["assign"][:50]).all()
    m = oracle.mti(X, C0, max_iters=15, history=True)
    np.testing.assert_array_equal(m["assign_hist"], r["assign_hist"])


def test_planted_clusters_reach_global_optimum():
    """Tiny planted data: Lloyd's from one seed per cluster reaches the optimum
    found by enumerating all k^n labelings."""
    rng = np.random.default_rng(21)
    for trial in range(6):
        k, per = 3, [3, 2, 3]
        centers = np.array([[0.0, 0.0], [9.0, 1.0], [2.0, 10.0]])
        X = np.concatenate([c + 0.6 * rng.standard_normal((p, 2)) for c, p in zip(centers, per)])
        X = X.astype(np.float32)
        n = X.shape[0]
        seeds = [0, per[0], per[0] + per[1]]
        r = oracle.lloyd(X, X[seeds].astype(np.float64), max_iters=50)
        Xd = X.astype(np.float64)
        best = np.inf
        best_lab = None
        for lab in itertools.product(range(k), repeat=n):
            lab = np.array(lab)
            if len(set(lab.tolist())) < k:
                continue
            sse = sum(((Xd[lab == j] - Xd[lab == j].mean(0)) ** 2).sum() for j in range(k))
            if sse < best - 1e-12:
                best, best_lab = sse, lab
        assert r["inertia"][-1] == pytest.approx(best, rel=1e-12)
        # same partition up to relabelling
        pairs = set(zip(r["assign"].tolist(), best_lab.tolist()))
        assert len(pairs) == k


# --------------------------------------------------------------------------- independent libraries


@pytest.mark.parametrize("seed,n,d,k", [(1, 2000, 2, 7), (2, 3000, 16, 10), (3, 1000, 32, 50)])
def test_assign_matches_scipy_vq(seed, n, d, k):
    from scipy.cluster.vq import vq
    X, C0 = synth.blobs(n, d, k, seed=seed, spread=3.0)
    Cm = C0.astype(np.float64) + 0.01
    a, best, second, _ = oracle.assign(X, Cm)
    codes, dist = vq(X.astype(np.float64), Cm)
    gap = (second - best) / np.maximum(second, 1e-300)
    sel = gap > 1e-12
    assert sel.mean() > 0.99
    np.testing.assert_array_equal(a[sel], codes[sel])
    # scipy may use the expanded form |x|^2 - 2x.c + |c|^2, which loses digits
    np.testing.assert_allclose(np.sqrt(best), dist, rtol=1e-9)


@pytest.mark.parametrize("seed,n,d,k,T", [(4, 4000, 3, 8, 30), (5, 3000, 16, 20, 40)])
def test_run_matches_sklearn_lloyd(seed, n, d, k, T):
    from sklearn.cluster import KMeans
    X, C0 = synth.blobs(n, d, k, seed=seed, spread=5.0)
    r = oracle.lloyd(X, C0, max_iters=T)
    counts = np.bincount(r["assign"], minlength=k)
    assert counts.min() > 0, "sklearn relocates empty clusters; pick data without them"
    km = KMeans(n_clusters=k, init=C0.astype(np.float64), n_init=1, max_iter=T, tol=0.0,
                algorithm="lloyd").fit(X.astype(np.float64))
    gap = (r["second"] - r["best"]) / r["second"]
    sel = gap > 1e-9
    np.testing.assert_array_equal(r["assign"][sel], km.labels_[sel])
    np.testing.assert_allclose(r["C"], km.cluster_centers_, rtol=1e-9, atol=1e-9)


# --------------------------------------------------------------------------- MTI reference


@pytest.mark.parametrize("seed,n,d,k,sigma", [
    (1, 3000, 2, 8, 1.0), (2, 2000, 16, 10, 1.0), (3, 2000, 8, 30, 3.0),
    (4, 1500, 3, 1, 1.0), (5, 2500, 32, 20, 6.0), (6, 1000, 1, 5, 2.0)])
def test_mti_equals_oracle_every_iteration(seed, n, d, k, sigma):
    X, C0 = synth.blobs(n, d, k, seed=seed, spread=5.0, sigma=sigma)
    r = oracle.lloyd(X, C0, max_iters=20, history=True)
    m = oracle.mti(X, C0, max_iters=20, history=True, check_bounds=True)
    assert m["iters"] == r["iters"]
    np.testing.assert_array_equal(m["assign_hist"], r["assign_hist"])
    np.testing.assert_array_equal(m["changed"], r["changed"])
    np.testing.assert_allclose(m["C"], r["C"], rtol=1e-12, atol=1e-12)
    assert m["bound_violations"] == 0
    assert (m["computed"] <= n * k).all()
    if k == 1:
        assert (m["clause1"][1:] == n).all()


def test_mti_prunes_on_separated_data():
    X, C0 = synth.blobs(5000, 8, 10, seed=8, spread=20.0, sigma=1.0)
    m = oracle.mti(X, C0, max_iters=20)
    frac = m["computed"][1:].sum() / (5000 * 10 * (m["iters"] - 1))
    assert frac < 0.2


def test_mti_tol_stopping_matches_oracle():
    X, C0 = synth.blobs(4000, 4, 9, seed=13, spread=4.0, sigma=1.5)
    for tol in (0.0, 0.001, 0.01, 0.05):
        r = oracle.lloyd(X, C0, max_iters=60, tol=tol)
        m = oracle.mti(X, C0, max_iters=60, tol=tol)
        assert r["iters"] == m["iters"]
        np.testing.assert_array_equal(m["assign"], r["assign"])


def test_negative_control_without_half_factor_fails():
    """Dropping the factor 1/2 from the clause thresholds (the literal reading
    of section III-C's clauses) must break the equality with the oracle."""
    # The one-dimensional counterexample: c_a = 0, c = 2, x = 1.5.  With the
    # full distance 2 as threshold, u = 1.5 <= 2 keeps x at c_a although
    # d(x, c) = 0.5.
    X = np.array([[-0.5], [0.5], [1.5], [2.0], [2.0], [2.0]], np.float32)
    C0 = np.array([[0.0], [2.5]])
    r = oracle.lloyd(X, C0, max_iters=4, history=True)
    good = oracle.mti(X, C0, max_iters=4, history=True)
    bad = oracle.mti(X, C0, max_iters=4, history=True, halve=False)
    np.testing.assert_array_equal(good["assign_hist"], r["assign_hist"])
    assert not np.array_equal(bad["assign_hist"], r["assign_hist"])
    # and on random overlapping mixtures the mistake shows up as well
    mismatches = 0
    for seed in range(10):
        X, C0 = synth.blobs(600, 2, 8, seed=100 + seed, spread=3.0, sigma=1.5)
        r = oracle.lloyd(X, C0, max_iters=10, history=True)
        bad = oracle.mti(X, C0, max_iters=10, history=True, halve=False)
        mismatches += int(not np.array_equal(bad["assign_hist"], r["assign_hist"]))
    assert mismatches > 0


def test_oracle_rejects_bad_arguments():
    X = np.zeros((4, 2), np.float32)
    with pytest.raises(ValueError):
        oracle.lloyd(X, np.zeros((5, 2)), 3)          # k > n
    with pytest.raises(ValueError):
        oracle.lloyd(X, np.zeros((2, 2)), 0)          # max_iters < 1
    with pytest.raises(ValueError):
        oracle.lloyd(X, np.zeros((2, 2)), 3, tol=-1.0)
    with pytest.raises(ValueError):
        oracle.lloyd(X, np.zeros((2, 3)), 3)          # shape mismatch
