"""ctypes loader for ``libkmeans_mti.so`` (the C ABI of include/kmeans_mti.h).

The library is required: there is no fallback.  Build it in-tree with
``python -m paper_1902_09527_amd.build``.
"""
from __future__ import annotations

import ctypes as C
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkmeans_mti.so")

KM_OK = 0
KM_ERR_INVALID_ARG = -1
KM_ERR_OOM = -2
KM_ERR_HIP = -3
KM_ERR_UNSUPPORTED = -4
KM_ERR_STATE = -5
KM_ERR_NONFINITE = -6

KM_FLAG_NO_PRUNE = 1
KM_FLAG_STATS = 2
KM_FLAG_VALIDATE = 4
KM_FLAG_TIMING = 8
KM_FLAG_VECTOR_ONLY = 16
KM_FLAG_LARGE_PATH = 32
KM_FLAG_GENERIC = 64
KM_FLAG_FULL_SUMS = 128
KM_FLAG_SPHERICAL = 256
KM_FLAG_ELKAN = 512

KM_PP_NO_PRUNE = 1
KM_PP_TIMING = 2

#: Every symbol include/kmeans_mti.h declares.
EXPORTS = (
    "kmeans_mti_init", "kmeans_mti_iterate", "kmeans_mti_get", "kmeans_mti_get_centroids64",
    "kmeans_mti_get_stats", "kmeans_mti_get_history", "kmeans_mti_get_timing", "kmeans_mti_run",
    "kmeans_mti_path", "kmeans_mti_destroy", "kmeans_mti_release_cache",
    "kmeans_mti_strerror", "kmeans_mti_last_hip_error",
    "kmeans_pp_workspace_bytes", "kmeans_pp_seed", "kmeans_pp_seed_noalloc", "kmeans_pp_run_best",
)

#: Size of the static workspace of kmeans_pp_seed_noalloc (KMEANS_PP_STATIC_WORKSPACE_BYTES).
KMEANS_PP_STATIC_WORKSPACE_BYTES = 64 << 20


class KmStats(C.Structure):
    _fields_ = [
        ("iterations", C.c_int32),
        ("converged", C.c_int32),
        ("changed_last", C.c_int64),
        ("dist_computed", C.c_int64),
        ("dist_lloyd", C.c_int64),
        ("clause1_skips", C.c_int64),
        ("rechecks", C.c_int64),
        ("inertia_last", C.c_double),
        ("device_ms", C.c_double),
    ]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_}


class KmPPStats(C.Structure):
    _fields_ = [
        ("computed", C.c_int64),
        ("improved", C.c_int64),
        ("passes", C.c_int32),
        ("pad_", C.c_int32),
        ("pass_ms", C.c_double),
        ("later_pass_ms", C.c_double),
        ("draw_ms", C.c_double),
    ]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_ if name != "pad_"}


class KMError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        msg = "%s failed: %s (%d)" % (where, _strerror(status), status)
        if detail:
            msg += ": " + detail
        super().__init__(msg)


_lib = None


def load() -> C.CDLL:
    """Load the HIP library once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libkmeans_mti.so not found at %s; build it with "
                          "`python -m paper_1902_09527_amd.build`" % LIB_PATH)
    lib = C.CDLL(LIB_PATH)
    P, i32, i64, u32, f64 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_double
    lib.kmeans_mti_init.argtypes = [C.POINTER(P), P, i64, i32, i32, P, P, u32]
    lib.kmeans_mti_init.restype = C.c_int
    lib.kmeans_mti_iterate.argtypes = [P, C.POINTER(i64)]
    lib.kmeans_mti_iterate.restype = C.c_int
    lib.kmeans_mti_get.argtypes = [P, P, P]
    lib.kmeans_mti_get.restype = C.c_int
    lib.kmeans_mti_get_centroids64.argtypes = [P, P]
    lib.kmeans_mti_get_centroids64.restype = C.c_int
    lib.kmeans_mti_get_stats.argtypes = [P, C.POINTER(KmStats)]
    lib.kmeans_mti_get_stats.restype = C.c_int
    lib.kmeans_mti_get_history.argtypes = [P, P, P, P, P, P, i32]
    lib.kmeans_mti_get_history.restype = C.c_int
    lib.kmeans_mti_get_timing.argtypes = [P, P, C.POINTER(i64)]
    lib.kmeans_mti_get_timing.restype = C.c_int
    lib.kmeans_mti_run.argtypes = [P, i64, i32, i32, P, i32, f64, P, P, P, u32, C.POINTER(KmStats)]
    lib.kmeans_mti_run.restype = C.c_int
    lib.kmeans_mti_path.argtypes = [P]
    lib.kmeans_mti_path.restype = C.c_char_p
    lib.kmeans_mti_destroy.argtypes = [P]
    lib.kmeans_mti_destroy.restype = None
    lib.kmeans_mti_release_cache.argtypes = []
    lib.kmeans_mti_release_cache.restype = None
    lib.kmeans_mti_strerror.argtypes = [C.c_int]
    lib.kmeans_mti_strerror.restype = C.c_char_p
    lib.kmeans_pp_workspace_bytes.argtypes = [i64, i32, i32]
    lib.kmeans_pp_workspace_bytes.restype = C.c_size_t
    lib.kmeans_pp_seed.argtypes = [P, i64, i32, i32, P, P, P, P, P, C.c_size_t, u32, P, C.POINTER(KmPPStats)]
    lib.kmeans_pp_seed.restype = C.c_int
    lib.kmeans_pp_seed_noalloc.argtypes = [P, i64, i32, i32, P, P, P, P, u32, P]
    lib.kmeans_pp_seed_noalloc.restype = C.c_int
    lib.kmeans_pp_run_best.argtypes = [P, i64, i32, i32, P, i32, i32, f64, P, P, P, u32, P, P,
                                       C.POINTER(KmStats)]
    lib.kmeans_pp_run_best.restype = C.c_int
    lib.kmeans_mti_last_hip_error.argtypes = []
    lib.kmeans_mti_last_hip_error.restype = C.c_char_p
    _lib = lib
    return lib


def _strerror(status: int) -> str:
    try:
        return load().kmeans_mti_strerror(status).decode()
    except ImportError:
        return "status %d" % status


def check(status: int, where: str) -> None:
    if status != KM_OK:
        detail = load().kmeans_mti_last_hip_error().decode()
        raise KMError(status, where, detail)
