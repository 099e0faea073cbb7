"""Seeded synthetic inputs for the k-means hot path.

This module draws data matrices X (n x d, float32, row-major) and initial
centroids C0 (k x d, float32) for the five benchmark workloads and for small
test cases.  It holds none of the clustering arithmetic: it only samples
Gaussian mixtures.  Both the CPU oracle (tests) and the GPU path (tests,
bench) take their inputs from here, so the two sides always see the same
bytes.

The paper measures on Friendster eigenvector embeddings (66M x 8 and
66M x 32) and on random matrices whose generator parameters it does not
give; none of those are available, so seeded mixtures of the same shape
class stand in for them (low-dimensional, clustered, most points stable).

Reproducibility: parameters come from the stream
``SeedSequence(ROOT_SEED, spawn_key=(workload_id, 0))``; rows are drawn in
chunks of ``CHUNK_ROWS`` rows, chunk ``c`` from
``SeedSequence(ROOT_SEED, spawn_key=(workload_id, 1, c))``, so any chunk can
be regenerated on its own and chunks can be drawn in parallel.  Values are
computed in float64 and stored as float32.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os
from typing import Dict, Optional, Tuple

import numpy as np

ROOT_SEED = 190209527
CHUNK_ROWS = 1 << 20


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: shape, mixture recipe and run settings."""

    name: str
    wid: int            # workload id, part of every seed
    n: int
    d: int
    k: int
    max_iters: int
    tol: float
    mixture: str        # "iso" or "aniso"
    mean_dist: str      # "uniform" or "normal"
    mean_scale: float   # half-width of U[-a, a] or std of N(0, a^2)
    sigma: Tuple[float, float]   # per-component isotropic std drawn U[lo, hi] (lo == hi: fixed)
    weights: str        # "equal", "dirichlet1" or "zipf1.1"
    noise_frac: float = 0.0

    @property
    def x_bytes(self) -> int:
        return self.n * self.d * 4


WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in [
        Workload("blobs-10k-d16-k8", 1, 10_000, 16, 8, 20, 0.0,
                 "iso", "uniform", 10.0, (1.0, 1.0), "equal"),
        Workload("blobs-1M-d32-k100", 2, 1_000_000, 32, 100, 30, 0.0,
                 "iso", "uniform", 20.0, (0.5, 2.0), "dirichlet1"),
        Workload("aniso-8M-d16-k10", 3, 8_000_000, 16, 10, 50, 0.001,
                 "aniso", "uniform", 10.0, (0.0, 0.0), "equal", noise_frac=0.05),
        Workload("blobs-2M-d256-k1000", 4, 2_000_000, 256, 1000, 20, 0.0,
                 "iso", "normal", 2.0, (1.0, 1.0), "equal"),
        Workload("zipf-100M-d32-k64", 5, 100_000_000, 32, 64, 25, 0.0,
                 "iso", "uniform", 50.0, (1.0, 5.0), "zipf1.1"),
    ]
}

#: Workload names in the order the benchmark table lists them.
ORDER = list(WORKLOADS)


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(ROOT_SEED, spawn_key=key)))


@dataclasses.dataclass
class MixtureParams:
    means: np.ndarray              # (m, d) float64
    weights: np.ndarray            # (m,) float64, sums to 1 (Gaussian components only)
    sigmas: Optional[np.ndarray]   # (m,) isotropic std, or None for anisotropic
    factors: Optional[np.ndarray]  # (m, d, d) x = mu + factor @ eps, or None for isotropic
    box_lo: Optional[np.ndarray]   # noise box (d,) or None
    box_hi: Optional[np.ndarray]


def mixture_params(w: Workload) -> MixtureParams:
    """Draw the mixture parameters of workload ``w`` from its parameter stream."""
    rng = _rng(w.wid, 0)
    m, d = w.k, w.d
    if w.mean_dist == "uniform":
        means = rng.uniform(-w.mean_scale, w.mean_scale, size=(m, d))
    else:
        means = rng.normal(0.0, w.mean_scale, size=(m, d))
    if w.weights == "equal":
        weights = np.full(m, 1.0 / m)
    elif w.weights == "dirichlet1":
        weights = rng.dirichlet(np.ones(m))
    elif w.weights == "zipf1.1":
        weights = np.arange(1, m + 1, dtype=np.float64) ** -1.1
        weights /= weights.sum()
    else:
        raise ValueError(w.weights)
    sigmas = factors = lo = hi = None
    if w.mixture == "iso":
        lo_s, hi_s = w.sigma
        sigmas = np.full(m, lo_s) if lo_s == hi_s else rng.uniform(lo_s, hi_s, size=m)
    else:
        factors = np.empty((m, d, d))
        for j in range(m):
            q, r = np.linalg.qr(rng.standard_normal((d, d)))
            q = q * np.sign(np.diag(r))[None, :]          # sign-fixed orthogonal factor
            scales = rng.lognormal(0.0, 0.5, size=d)
            factors[j] = q * scales[None, :]               # R_j diag(s_j)
        if w.noise_frac > 0:
            # Noise box: per-dimension 3-sigma envelope of all components.
            std = np.sqrt((factors ** 2).sum(axis=2))      # (m, d) per-dim std of each component
            lo = (means - 3.0 * std).min(axis=0)
            hi = (means + 3.0 * std).max(axis=0)
    return MixtureParams(means, weights, sigmas, factors, lo, hi)


def _fill_chunk(w: Workload, p: MixtureParams, c: int, out: np.ndarray) -> None:
    rows = out.shape[0]
    rng = _rng(w.wid, 1, c)
    m = w.k
    if w.noise_frac > 0:
        probs = np.concatenate([p.weights * (1.0 - w.noise_frac), [w.noise_frac]])
        z = rng.choice(m + 1, size=rows, p=probs)
    else:
        z = rng.choice(m, size=rows, p=p.weights)
    eps = rng.standard_normal((rows, w.d))
    if p.sigmas is not None:
        x = p.means[z] + eps * p.sigmas[z][:, None]
    else:
        x = np.empty((rows, w.d))
        for j in range(m):
            sel = z == j
            x[sel] = p.means[j] + eps[sel] @ p.factors[j].T
    if w.noise_frac > 0:
        sel = z == m
        u = rng.random((int(sel.sum()), w.d))
        x[sel] = p.box_lo + (p.box_hi - p.box_lo) * u
    out[:] = x.astype(np.float32)


def make_x(w: Workload, n: Optional[int] = None, threads: Optional[int] = None) -> np.ndarray:
    """Rows [0, n) of workload ``w`` (default: all rows) as float32 (n, d)."""
    n = w.n if n is None else min(n, w.n)
    p = mixture_params(w)
    X = np.empty((n, w.d), dtype=np.float32)
    nchunks = (n + CHUNK_ROWS - 1) // CHUNK_ROWS

    def job(c: int) -> None:
        lo = c * CHUNK_ROWS
        hi = min(n, lo + CHUNK_ROWS)
        if hi - lo == CHUNK_ROWS or hi == w.n:
            _fill_chunk(w, p, c, X[lo:hi])
        else:   # a prefix ending inside a chunk: draw the whole chunk, keep its head
            tmp = np.empty((min(CHUNK_ROWS, w.n - lo), w.d), dtype=np.float32)
            _fill_chunk(w, p, c, tmp)
            X[lo:hi] = tmp[: hi - lo]

    threads = threads or min(16, os.cpu_count() or 1)
    if nchunks == 1 or threads == 1:
        for c in range(nchunks):
            job(c)
    else:
        with _cf.ThreadPoolExecutor(threads) as ex:
            list(ex.map(job, range(nchunks)))
    return X


def seed_indices(w: Workload, X: np.ndarray) -> np.ndarray:
    """k distinct row indices of X chosen by the workload's parameter stream.

    Draws without replacement and redraws until the chosen rows are pairwise
    distinct as float32 vectors.
    """
    rng = _rng(w.wid, 2)
    n = X.shape[0]
    for _ in range(100):
        idx = rng.choice(n, size=w.k, replace=False)
        rows = np.ascontiguousarray(X[idx])
        if np.unique(rows, axis=0).shape[0] == w.k:
            return idx
    raise RuntimeError("could not draw k distinct seed rows")


def make(name: str, n: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray, Workload]:
    """X (n, d) float32, C0 (k, d) float32 and the workload record.

    With ``n`` smaller than the workload's size, X is the first ``n`` rows and
    C0 is still drawn from those rows.
    """
    w = WORKLOADS[name]
    X = make_x(w, n)
    idx = seed_indices(w, X)
    return X, np.ascontiguousarray(X[idx]), w


def blobs(n: int, d: int, k: int, seed: int, spread: float = 10.0, sigma: float = 1.0,
          comps: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray]:
    """A small isotropic Gaussian mixture for tests: X (n, d), C0 (k, d) float32.

    ``comps`` mixture components (default k) with means U[-spread, spread]^d
    and std ``sigma``; C0 = k distinct rows of X chosen by the same seed.
    """
    rng = _rng(1000, seed)
    m = comps or k
    means = rng.uniform(-spread, spread, size=(m, d))
    z = rng.integers(0, m, size=n)
    X = (means[z] + sigma * rng.standard_normal((n, d))).astype(np.float32)
    for _ in range(100):
        idx = rng.choice(n, size=k, replace=False)
        C0 = np.ascontiguousarray(X[idx])
        if np.unique(C0, axis=0).shape[0] == k:
            return X, C0
    raise RuntimeError("could not draw k distinct seed rows")
