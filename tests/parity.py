"""Comparison rules between the GPU path and the CPU oracle.

The bar: assignments identical wherever the oracle's best-vs-second relative
gap (D2 - D1) / D2 of squared distances exceeds 1e-5; centroids within 1e-5
relative, per centroid, ||c_gpu - c_ref|| <= 1e-5 * max(||c_ref||, rms row
norm of X) (per-coordinate relative error is ill-posed near zero); identical
iteration counts.
"""
import numpy as np

GAP = 1e-5
CTOL = 1e-5


def rel_gap(best: np.ndarray, second: np.ndarray) -> np.ndarray:
    with np.errstate(divide="ignore", invalid="ignore"):
        g = (second - best) / second
    g = np.where(np.isinf(second), 1.0, g)
    g = np.where(second == 0, 0.0, g)
    return g


def check_assign(a_gpu: np.ndarray, a_ref: np.ndarray, best: np.ndarray, second: np.ndarray,
                 what: str = "") -> dict:
    gap = rel_gap(best, second)
    mism = a_gpu != a_ref
    bad = mism & (gap > GAP)
    assert not bad.any(), "%s: %d assignments differ at gap > %g (first rows %s)" % (
        what, int(bad.sum()), GAP, np.nonzero(bad)[0][:10].tolist())
    return {"mismatch": int(mism.sum()), "near_ties": int((gap <= GAP).sum())}


def check_centroids(C_gpu: np.ndarray, C_ref: np.ndarray, X: np.ndarray, what: str = "",
                    tol: float = CTOL) -> float:
    C_gpu = np.asarray(C_gpu, np.float64)
    C_ref = np.asarray(C_ref, np.float64)
    rms = float(np.sqrt(np.mean(np.sum(X.astype(np.float64) ** 2, axis=1)))) if len(X) else 0.0
    err = np.linalg.norm(C_gpu - C_ref, axis=1)
    scale = np.maximum(np.linalg.norm(C_ref, axis=1), rms)
    rel = err / np.where(scale > 0, scale, 1.0)
    worst = float(rel.max()) if rel.size else 0.0
    assert worst <= tol, "%s: centroid relative error %.3g > %g (cluster %d)" % (
        what, worst, tol, int(rel.argmax()))
    return worst
