"""Python binding of the MTI k-means C ABI (include/kmeans_mti.h).

Argument marshalling only: tensors are checked (device, dtype, shape,
contiguity) and their device pointers and the current HIP stream are handed
to ``libkmeans_mti.so``; every step of the computation runs in its kernels.
PyTorch provides device memory and streams.
"""
from __future__ import annotations

import ctypes as C
from typing import Dict, Optional, Tuple

import numpy as np
import torch

from . import _native as N


def _check_matrix(t: torch.Tensor, name: str, cols: Optional[int] = None) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.device.type != "cuda":
        raise ValueError("%s must be on a GPU device, got %s" % (name, t.device))
    if t.dtype != torch.float32:
        raise ValueError("%s must be float32, got %s" % (name, t.dtype))
    if t.dim() != 2:
        raise ValueError("%s must be 2-D" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous (row-major)" % name)
    if cols is not None and t.shape[1] != cols:
        raise ValueError("%s must have %d columns" % (name, cols))


def _flags(prune: bool, stats: bool, validate: bool, timing: bool = False,
           vector_only: bool = False, large_path: bool = False, generic: bool = False,
           full_sums: bool = False, spherical: bool = False, elkan: bool = False) -> int:
    f = N.KM_FLAG_TIMING if timing else 0
    if elkan:
        f |= N.KM_FLAG_ELKAN
    if spherical:
        f |= N.KM_FLAG_SPHERICAL
    if full_sums:
        f |= N.KM_FLAG_FULL_SUMS
    if generic:
        f |= N.KM_FLAG_GENERIC
    if vector_only:
        f |= N.KM_FLAG_VECTOR_ONLY
    if large_path:
        f |= N.KM_FLAG_LARGE_PATH
    if not prune:
        f |= N.KM_FLAG_NO_PRUNE
    if stats:
        f |= N.KM_FLAG_STATS
    if validate:
        f |= N.KM_FLAG_VALIDATE
    return f


def _stream_ptr(device: torch.device, stream: Optional[torch.cuda.Stream]) -> C.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return C.c_void_p(s.cuda_stream)


class KMeansMTI:
    """One k-means problem on the GPU (wraps kmeans_mti_init / iterate / get).

    X (n x d float32, contiguous, on the GPU) is borrowed for the lifetime of
    the object and must not change; C0 (k x d) is copied at construction.
    """

    def __init__(self, X: torch.Tensor, C0: torch.Tensor, prune: bool = True, stats: bool = False,
                 validate: bool = False, timing: bool = False, vector_only: bool = False,
                 large_path: bool = False, generic: bool = False, full_sums: bool = False,
                 spherical: bool = False, elkan: bool = False, stream: Optional[torch.cuda.Stream] = None):
        _check_matrix(X, "X")
        _check_matrix(C0, "C0", X.shape[1])
        if C0.device != X.device:
            raise ValueError("X and C0 must be on the same device")
        self._lib = N.load()
        self.X = X
        self.n, self.d = X.shape
        self.k = C0.shape[0]
        self.device = X.device
        self.stream = stream
        self._ctx = C.c_void_p()
        with torch.cuda.device(self.device):
            st = self._lib.kmeans_mti_init(C.byref(self._ctx), C.c_void_p(X.data_ptr()), self.n,
                                           self.d, self.k, C.c_void_p(C0.data_ptr()),
                                           _stream_ptr(self.device, stream),
                                           _flags(prune, stats, validate, timing, vector_only,
                                                  large_path, generic, full_sums, spherical, elkan))
        N.check(st, "kmeans_mti_init")

    def _live(self) -> C.c_void_p:
        if not self._ctx:
            raise RuntimeError("context is closed")
        return self._ctx

    def iterate(self, sync: bool = False) -> Optional[int]:
        """Enqueue one iteration; with sync=True wait and return the changed count."""
        ch = C.c_int64(0)
        with torch.cuda.device(self.device):
            st = self._lib.kmeans_mti_iterate(self._live(), C.byref(ch) if sync else None)
        N.check(st, "kmeans_mti_iterate")
        return int(ch.value) if sync else None

    def get(self, assign: bool = True, centroids: bool = True
            ) -> Tuple[Optional[torch.Tensor], Optional[torch.Tensor]]:
        """Current assignment (int32 [n]) and float32 centroids ([k, d])."""
        a = torch.empty(self.n, dtype=torch.int32, device=self.device) if assign else None
        c = torch.empty(self.k, self.d, dtype=torch.float32, device=self.device) if centroids else None
        with torch.cuda.device(self.device):
            st = self._lib.kmeans_mti_get(self._live(), C.c_void_p(a.data_ptr()) if a is not None else None,
                                          C.c_void_p(c.data_ptr()) if c is not None else None)
        N.check(st, "kmeans_mti_get")
        return a, c

    def centroids64(self) -> np.ndarray:
        """float64 master centroids (host copy, [k, d])."""
        out = np.empty((self.k, self.d), np.float64)
        with torch.cuda.device(self.device):
            st = self._lib.kmeans_mti_get_centroids64(self._live(), out.ctypes.data_as(C.c_void_p))
        N.check(st, "kmeans_mti_get_centroids64")
        return out

    def stats(self) -> Dict[str, float]:
        s = N.KmStats()
        with torch.cuda.device(self.device):
            st = self._lib.kmeans_mti_get_stats(self._live(), C.byref(s))
        N.check(st, "kmeans_mti_get_stats")
        return s.as_dict()

    def history(self, cap: int = 4096) -> Dict[str, np.ndarray]:
        """Per-iteration changed / computed / clause1 / rechecks / inertia."""
        arrs = {name: np.zeros(cap, np.int64) for name in ("changed", "computed", "clause1", "rechecks")}
        arrs["inertia"] = np.zeros(cap, np.float64)
        p = lambda a: a.ctypes.data_as(C.c_void_p)
        with torch.cuda.device(self.device):
            m = self._lib.kmeans_mti_get_history(self._live(), p(arrs["changed"]), p(arrs["computed"]),
                                                 p(arrs["clause1"]), p(arrs["rechecks"]),
                                                 p(arrs["inertia"]), cap)
        if m < 0:
            N.check(m, "kmeans_mti_get_history")
        return {name: a[:m] for name, a in arrs.items()}

    def path(self) -> str:
        """Kernel path of this context (kmeans_mti_path)."""
        return self._lib.kmeans_mti_path(self._live()).decode()

    def timing(self) -> Dict[str, float]:
        """Per-kernel device milliseconds (HIP events) over the iterations so far."""
        ms = (C.c_double * 4)()
        it = C.c_int64(0)
        with torch.cuda.device(self.device):
            st = self._lib.kmeans_mti_get_timing(self._live(), ms, C.byref(it))
        N.check(st, "kmeans_mti_get_timing")
        return {"assign_ms": ms[0], "reduce_ms": ms[1], "update_ms": ms[2], "table_ms": ms[3],
                "iters": int(it.value)}

    def close(self) -> None:
        if self._ctx:
            self._lib.kmeans_mti_destroy(self._ctx)
            self._ctx = C.c_void_p()

    def __enter__(self) -> "KMeansMTI":
        return self

    def __exit__(self, *exc) -> None:
        self.close()

    def __del__(self) -> None:
        try:
            self.close()
        except Exception:
            pass


def run(X: torch.Tensor, C0: torch.Tensor, max_iters: int, tol: float = 0.0, prune: bool = True,
        stats: bool = False, validate: bool = False, vector_only: bool = False,
        large_path: bool = False, generic: bool = False, full_sums: bool = False,
        spherical: bool = False, elkan: bool = False, stream: Optional[torch.cuda.Stream] = None
        ) -> Tuple[torch.Tensor, torch.Tensor, Dict[str, float]]:
    """Whole k-means run (kmeans_mti_run): (assign int32 [n], C float32 [k, d], stats)."""
    _check_matrix(X, "X")
    _check_matrix(C0, "C0", X.shape[1])
    if C0.device != X.device:
        raise ValueError("X and C0 must be on the same device")
    lib = N.load()
    n, d = X.shape
    k = C0.shape[0]
    a = torch.empty(n, dtype=torch.int32, device=X.device)
    c = torch.empty(k, d, dtype=torch.float32, device=X.device)
    s = N.KmStats()
    with torch.cuda.device(X.device):
        st = lib.kmeans_mti_run(C.c_void_p(X.data_ptr()), n, d, k, C.c_void_p(C0.data_ptr()),
                                int(max_iters), float(tol), C.c_void_p(a.data_ptr()),
                                C.c_void_p(c.data_ptr()), _stream_ptr(X.device, stream),
                                _flags(prune, stats, validate, False, vector_only, large_path,
                                       generic, full_sums, spherical, elkan),
                                C.byref(s))
    N.check(st, "kmeans_mti_run")
    return a, c, s.as_dict()


def kmeanspp(X: torch.Tensor, k: int, u, prune: bool = True, count: bool = False, timing: bool = False,
             workspace: Optional[torch.Tensor] = None, stream: Optional[torch.cuda.Stream] = None
             ) -> Dict[str, object]:
    """k-means++ seeding (kmeans_pp_seed) of k rows of X with the uniforms u.

    u: k floats in [0, 1) (host).  Returns ``C`` (float32 [k, d], the seed
    rows in draw order), ``idx`` (int64 [k]) and ``D2`` (float64 [n], squared
    distance of each row to its nearest seed), all on X's device, and with
    ``count`` or ``timing`` also ``stats`` (km_pp_stats as a dict: distances
    computed, rows improved, and with ``timing`` the device milliseconds of
    the passes and the draws; synchronizes).
    ``workspace``: optional uint8 device tensor of at least
    :func:`kmeanspp_workspace_bytes` bytes, reused across calls.
    """
    _check_matrix(X, "X")
    lib = N.load()
    n, d = X.shape
    k = int(k)
    uu = np.ascontiguousarray(np.asarray(u, dtype=np.float64).reshape(-1))
    if uu.shape != (k,):
        raise ValueError("u must hold k = %d uniforms" % k)
    need = int(lib.kmeans_pp_workspace_bytes(n, d, k))
    if need == 0:
        raise N.KMError(N.KM_ERR_INVALID_ARG, "kmeans_pp_workspace_bytes")
    if workspace is None:
        workspace = torch.empty(need + 256, dtype=torch.uint8, device=X.device)
    if workspace.device != X.device or workspace.dtype != torch.uint8 or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 tensor on X's device")
    off = (-workspace.data_ptr()) % 256
    if workspace.numel() - off < need:
        raise ValueError("workspace needs %d bytes (256-byte aligned)" % need)
    c = torch.empty(k, d, dtype=torch.float32, device=X.device)
    idx = torch.empty(k, dtype=torch.int64, device=X.device)
    d2 = torch.empty(n, dtype=torch.float64, device=X.device)
    ps = N.KmPPStats()
    flags = (0 if prune else N.KM_PP_NO_PRUNE) | (N.KM_PP_TIMING if timing else 0)
    with torch.cuda.device(X.device):
        st = lib.kmeans_pp_seed(C.c_void_p(X.data_ptr()), n, d, k, uu.ctypes.data_as(C.c_void_p),
                                C.c_void_p(c.data_ptr()), C.c_void_p(idx.data_ptr()),
                                C.c_void_p(d2.data_ptr()), C.c_void_p(workspace.data_ptr() + off),
                                workspace.numel() - off, flags, _stream_ptr(X.device, stream),
                                C.byref(ps) if (count or timing) else None)
    N.check(st, "kmeans_pp_seed")
    out = {"C": c, "idx": idx, "D2": d2}
    if count or timing:
        out["stats"] = ps.as_dict()
    return out


def kmeanspp_noalloc(X: torch.Tensor, k: int, u, prune: bool = True,
                     stream: Optional[torch.cuda.Stream] = None) -> Dict[str, object]:
    """k-means++ seeding with the library's static device workspace
    (kmeans_pp_seed_noalloc): the library allocates nothing.  Returns ``C``,
    ``idx`` and ``D2`` as :func:`kmeanspp` (those outputs are allocated here,
    by the caller's side)."""
    _check_matrix(X, "X")
    lib = N.load()
    n, d = X.shape
    k = int(k)
    uu = np.ascontiguousarray(np.asarray(u, dtype=np.float64).reshape(-1))
    if uu.shape != (k,):
        raise ValueError("u must hold k = %d uniforms" % k)
    c = torch.empty(k, d, dtype=torch.float32, device=X.device)
    idx = torch.empty(k, dtype=torch.int64, device=X.device)
    d2 = torch.empty(n, dtype=torch.float64, device=X.device)
    with torch.cuda.device(X.device):
        st = lib.kmeans_pp_seed_noalloc(C.c_void_p(X.data_ptr()), n, d, k, uu.ctypes.data_as(C.c_void_p),
                                        C.c_void_p(c.data_ptr()), C.c_void_p(idx.data_ptr()),
                                        C.c_void_p(d2.data_ptr()), 0 if prune else N.KM_PP_NO_PRUNE,
                                        _stream_ptr(X.device, stream))
    N.check(st, "kmeans_pp_seed_noalloc")
    return {"C": c, "idx": idx, "D2": d2}


def release_cache() -> None:
    """Free the device buffers the library keeps from released contexts
    (kmeans_mti_release_cache)."""
    N.load().kmeans_mti_release_cache()


def kmeanspp_workspace_bytes(n: int, d: int, k: int) -> int:
    """Bytes of workspace kmeans_pp_seed needs (plus up to 255 for alignment)."""
    return int(N.load().kmeans_pp_workspace_bytes(int(n), int(d), int(k)))


def run_pp_best(X: torch.Tensor, k: int, U, max_iters: int, tol: float = 0.0, prune: bool = True,
                stream: Optional[torch.cuda.Stream] = None) -> Dict[str, object]:
    """The paper's k-means++ with r restarts (kmeans_pp_run_best): for each
    row of U (r x k uniforms) seed with k-means++ and run k-means from the
    seeds; the library keeps the run with the least final inertia (ties: the
    earlier run).

    Returns ``best`` (the kept run's index), ``assign``, ``C``, ``stats`` of
    that run and ``inertia`` (every run's final inertia).
    """
    _check_matrix(X, "X")
    U = np.ascontiguousarray(np.asarray(U, dtype=np.float64))
    if U.ndim != 2 or U.shape[1] != int(k):
        raise ValueError("U must be r x k")
    lib = N.load()
    n, d = X.shape
    k = int(k)
    r = U.shape[0]
    a = torch.empty(n, dtype=torch.int32, device=X.device)
    c = torch.empty(k, d, dtype=torch.float32, device=X.device)
    best = C.c_int32(-1)
    inertia = np.zeros(r, np.float64)
    s = N.KmStats()
    with torch.cuda.device(X.device):
        st = lib.kmeans_pp_run_best(C.c_void_p(X.data_ptr()), n, d, k, U.ctypes.data_as(C.c_void_p), r,
                                    int(max_iters), float(tol), C.c_void_p(a.data_ptr()),
                                    C.c_void_p(c.data_ptr()), _stream_ptr(X.device, stream),
                                    _flags(prune, False, False), C.byref(best),
                                    inertia.ctypes.data_as(C.c_void_p), C.byref(s))
    N.check(st, "kmeans_pp_run_best")
    return {"best": int(best.value), "assign": a, "C": c, "stats": s.as_dict(), "inertia": inertia.tolist()}
