"""CPU oracle for the k-means hot path -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the package smoke check and the benchmark's CPU-baseline
leg may import this module.  The GPU library shares no code with it; nothing
in the product path imports it.

``lloyd`` / ``assign`` / ``update`` wrap plain float64 Lloyd's k-means (no
pruning) from ``lloyd.c``; ``mti`` wraps the separately written float64 MTI
reference from ``mti_ref.c``; ``spherical`` wraps float64 spherical k-means
(cosine proximity on the unit sphere) from ``spherical.c``; ``kmeanspp`` wraps
k-means++ seeding with caller-drawn uniforms from ``kmeanspp.c``.  All are compiled
with gcc into ``liboracle.so`` next to this file by :func:`build`.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SOURCES = [os.path.join(_HERE, "lloyd.c"), os.path.join(_HERE, "mti_ref.c"), os.path.join(_HERE, "spherical.c"),
           os.path.join(_HERE, "kmeanspp.c")]

_lib = None


def build(verbose: bool = False) -> str:
    """Compile the oracle with gcc (-O3, OpenMP, no fast-math, no FMA contraction)."""
    tmp = LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O3", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-Wall", "-Wextra", "-o", tmp] + SOURCES + ["-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    global _lib
    _lib = None
    return LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        build()
    lib = C.CDLL(LIB_PATH)
    P = C.c_void_p
    i64, i32, f64 = C.c_int64, C.c_int32, C.c_double
    lib.oracle_set_threads.argtypes = [i32]
    lib.oracle_set_threads.restype = None
    lib.oracle_get_threads.argtypes = []
    lib.oracle_get_threads.restype = i32
    lib.oracle_assign.argtypes = [P, i64, i32, P, i32, P, P, P, P]
    lib.oracle_assign.restype = i64
    lib.oracle_update.argtypes = [P, i64, i32, P, i32, P, P, P]
    lib.oracle_update.restype = i32
    lib.oracle_lloyd.argtypes = [P, i64, i32, i32, P, i32, f64, P, P, P, P, P, P, P, P, P]
    lib.oracle_lloyd.restype = i32
    lib.mti_lloyd.argtypes = [P, i64, i32, i32, P, i32, f64, i32, P, P, P, P, P, P, P, P]
    lib.mti_lloyd.restype = i32
    lib.oracle_spherical.argtypes = [P, i64, i32, i32, P, i32, f64, P, P, P, P, P, P, P]
    lib.oracle_spherical.restype = i32
    lib.oracle_kmeanspp.argtypes = [P, i64, i32, i32, P, P, P]
    lib.oracle_kmeanspp.restype = i32
    _lib = lib
    return lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _x(X: np.ndarray) -> np.ndarray:
    X = np.ascontiguousarray(X, dtype=np.float32)
    if X.ndim != 2:
        raise ValueError("X must be 2-D")
    return X


def _c(C0: np.ndarray, k: int, d: int) -> np.ndarray:
    C0 = np.ascontiguousarray(C0, dtype=np.float64)
    if C0.shape != (k, d):
        raise ValueError("centroids must be (k, d)")
    return C0


def set_threads(t: int) -> None:
    _load().oracle_set_threads(int(t))


def get_threads() -> int:
    return int(_load().oracle_get_threads())


def assign(X: np.ndarray, Cmat: np.ndarray, prev: Optional[np.ndarray] = None):
    """One assignment step: (a int32[n], best float64[n], second float64[n], changed)."""
    X = _x(X)
    n, d = X.shape
    Cm = np.ascontiguousarray(Cmat, dtype=np.float64)
    k = Cm.shape[0]
    if Cm.shape != (k, d):
        raise ValueError("centroids must be (k, d)")
    out = np.empty(n, np.int32)
    b = np.empty(n, np.float64)
    s = np.empty(n, np.float64)
    pv = None if prev is None else np.ascontiguousarray(prev, dtype=np.int32)
    ch = _load().oracle_assign(_ptr(X), n, d, _ptr(Cm), k, _ptr(pv), _ptr(out), _ptr(b), _ptr(s))
    return out, b, s, int(ch)


def update(X: np.ndarray, a: np.ndarray, C_old: np.ndarray):
    """One update step: (C_new float64[k, d], counts int64[k])."""
    X = _x(X)
    n, d = X.shape
    Co = np.ascontiguousarray(C_old, dtype=np.float64)
    k = Co.shape[0]
    a = np.ascontiguousarray(a, dtype=np.int32)
    if a.shape != (n,) or (n and (a.min() < 0 or a.max() >= k)):
        raise ValueError("assignment out of range")
    Cn = np.empty_like(Co)
    cnt = np.empty(k, np.int64)
    if _load().oracle_update(_ptr(X), n, d, _ptr(a), k, _ptr(Co), _ptr(Cn), _ptr(cnt)) != 0:
        raise MemoryError("oracle_update")
    return Cn, cnt


def lloyd(X: np.ndarray, C0: np.ndarray, max_iters: int, tol: float = 0.0,
          history: bool = False) -> Dict[str, np.ndarray]:
    """Plain float64 Lloyd's k-means from C0.

    Returns a dict with ``assign`` (int32[n], last step), ``C`` (float64[k, d],
    after the last update), ``iters``, ``inertia`` and ``changed`` (per
    iteration), ``best`` / ``second`` (last step's smallest and second-smallest
    squared distances), and with ``history`` also ``assign_hist``
    (iters x n) and ``C_hist`` (iters + 1 x k x d).
    """
    X = _x(X)
    n, d = X.shape
    k = np.asarray(C0).shape[0]
    C0 = _c(C0, k, d)
    T = int(max_iters)
    a = np.empty(n, np.int32)
    Cout = np.empty((k, d), np.float64)
    it = C.c_int32(0)
    J = np.zeros(T, np.float64)
    ch = np.zeros(T, np.int64)
    b = np.empty(n, np.float64)
    s = np.empty(n, np.float64)
    ah = np.empty((T, n), np.int32) if history else None
    chh = np.empty((T + 1, k, d), np.float64) if history else None
    rc = _load().oracle_lloyd(_ptr(X), n, d, k, _ptr(C0), T, float(tol), _ptr(a), _ptr(Cout),
                              C.byref(it), _ptr(J), _ptr(ch), _ptr(b), _ptr(s), _ptr(ah), _ptr(chh))
    if rc != 0:
        raise ValueError("oracle_lloyd rejected its arguments")
    t = it.value
    res = dict(assign=a, C=Cout, iters=t, inertia=J[:t], changed=ch[:t], best=b, second=s)
    if history:
        res["assign_hist"] = ah[:t]
        res["C_hist"] = chh[: t + 1]
    return res


def mti(X: np.ndarray, C0: np.ndarray, max_iters: int, tol: float = 0.0, halve: bool = True,
        history: bool = False, check_bounds: bool = False) -> Dict[str, np.ndarray]:
    """float64 MTI-pruned Lloyd's (CPU reference); ``halve=False`` is the negative control."""
    X = _x(X)
    n, d = X.shape
    k = np.asarray(C0).shape[0]
    C0 = _c(C0, k, d)
    T = int(max_iters)
    a = np.empty(n, np.int32)
    Cout = np.empty((k, d), np.float64)
    it = C.c_int32(0)
    ch = np.zeros(T, np.int64)
    comp = np.zeros(T, np.int64)
    c1 = np.zeros(T, np.int64)
    ah = np.empty((T, n), np.int32) if history else None
    bv = C.c_int64(0)
    rc = _load().mti_lloyd(_ptr(X), n, d, k, _ptr(C0), T, float(tol), int(bool(halve)), _ptr(a),
                           _ptr(Cout), C.byref(it), _ptr(ch), _ptr(comp), _ptr(c1), _ptr(ah),
                           C.byref(bv) if check_bounds else None)
    if rc != 0:
        raise ValueError("mti_lloyd rejected its arguments")
    t = it.value
    res = dict(assign=a, C=Cout, iters=t, changed=ch[:t], computed=comp[:t], clause1=c1[:t])
    if history:
        res["assign_hist"] = ah[:t]
    if check_bounds:
        res["bound_violations"] = int(bv.value)
    return res


def spherical(X: np.ndarray, C0: np.ndarray, max_iters: int, tol: float = 0.0) -> Dict[str, np.ndarray]:
    """float64 spherical k-means from C0 (rows of C0 nonzero).

    Returns ``assign``, ``C`` (unit centroids after the last update),
    ``iters``, ``objective`` (sum of squared chord distances 2 - 2 cos per
    step), ``changed``, and ``best`` / ``second`` (last step's smallest and
    second-smallest squared chord distances).
    """
    X = _x(X)
    n, d = X.shape
    k = np.asarray(C0).shape[0]
    C0 = _c(C0, k, d)
    T = int(max_iters)
    a = np.empty(n, np.int32)
    Cout = np.empty((k, d), np.float64)
    it = C.c_int32(0)
    J = np.zeros(T, np.float64)
    ch = np.zeros(T, np.int64)
    b = np.empty(n, np.float64)
    s = np.empty(n, np.float64)
    rc = _load().oracle_spherical(_ptr(X), n, d, k, _ptr(C0), T, float(tol), _ptr(a), _ptr(Cout),
                                  C.byref(it), _ptr(J), _ptr(ch), _ptr(b), _ptr(s))
    if rc != 0:
        raise ValueError("oracle_spherical rejected its arguments")
    t = it.value
    return dict(assign=a, C=Cout, iters=t, objective=J[:t], changed=ch[:t], best=b, second=s)


def kmeanspp(X: np.ndarray, k: int, u: np.ndarray) -> Dict[str, np.ndarray]:
    """k-means++ seeding of k rows of X with the uniforms u[0..k-1] in [0, 1).

    Returns ``idx`` (int64[k], seed row indices in draw order), ``C`` (the
    seed rows, float32[k, d]) and ``D2`` (float64[n], squared distance of each
    row to its nearest seed).
    """
    X = _x(X)
    n, d = X.shape
    u = np.ascontiguousarray(u, dtype=np.float64)
    if u.shape != (int(k),):
        raise ValueError("u must hold k uniforms")
    idx = np.empty(int(k), np.int64)
    D2 = np.empty(n, np.float64)
    if _load().oracle_kmeanspp(_ptr(X), n, d, int(k), _ptr(u), _ptr(idx), _ptr(D2)) != 0:
        raise ValueError("oracle_kmeanspp rejected its arguments")
    return dict(idx=idx, C=X[idx].copy(), D2=D2)
