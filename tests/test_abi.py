"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every entry point include/kmeans_mti.h declares, and rejects bad arguments
before it touches the device."""
import ctypes as C
import math
import os
import re

import pytest

from paper_1902_09527_amd import _native as N

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kmeans_mti.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kmeans_(?:mti|pp)_\w+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert _declared() == sorted(N.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = N.load()
    for name in _declared():
        assert hasattr(lib, name), name
        assert C.cast(getattr(lib, name), C.c_void_p).value


def test_status_texts():
    lib = N.load()
    for st in (N.KM_OK, N.KM_ERR_INVALID_ARG, N.KM_ERR_OOM, N.KM_ERR_HIP, N.KM_ERR_UNSUPPORTED,
               N.KM_ERR_STATE, N.KM_ERR_NONFINITE):
        txt = lib.kmeans_mti_strerror(st).decode()
        assert txt and txt != "unknown status"
    assert lib.kmeans_mti_strerror(12345).decode() == "unknown status"
    assert isinstance(lib.kmeans_mti_last_hip_error(), bytes)


def test_path_of_null_context_is_empty():
    assert N.load().kmeans_mti_path(None) == b""


def test_pp_stats_layout():
    assert C.sizeof(N.KmPPStats) == 48


def test_struct_layout_matches_header():
    # int32 x2, int64 x5, double x2 with natural alignment
    assert C.sizeof(N.KmStats) == 4 * 2 + 8 * 5 + 8 * 2


def test_init_rejects_bad_arguments_without_a_device():
    lib = N.load()
    fake = C.c_void_p(0x1000)   # never dereferenced: the shape checks fail first
    ctx = C.c_void_p()
    assert lib.kmeans_mti_init(None, fake, 10, 2, 2, fake, None, 0) == N.KM_ERR_INVALID_ARG
    cases = [
        (None, 10, 2, 2, fake),          # X null
        (fake, 10, 2, 2, None),          # C0 null
        (fake, 0, 2, 1, fake),           # n < 1
        (fake, 10, 0, 2, fake),          # d < 1
        (fake, 10, 2, 0, fake),          # k < 1
        (fake, 10, 2, 11, fake),         # k > n
        (fake, 2 ** 62, 4, 2, fake),     # n*d*4 overflows
    ]
    for X, n, d, k, C0 in cases:
        assert lib.kmeans_mti_init(C.byref(ctx), X, n, d, k, C0, None, 0) == N.KM_ERR_INVALID_ARG
        assert not ctx.value
    # unknown flag bits
    assert lib.kmeans_mti_init(C.byref(ctx), fake, 10, 2, 2, fake, None, 1 << 10) == N.KM_ERR_INVALID_ARG


def test_run_rejects_bad_arguments_without_a_device():
    lib = N.load()
    fake = C.c_void_p(0x1000)
    st = N.KmStats()
    good = dict(X=fake, n=10, d=2, k=2, C0=fake, it=5, tol=0.0, a=fake, c=fake)

    def call(**kw):
        a = dict(good, **kw)
        return lib.kmeans_mti_run(a["X"], a["n"], a["d"], a["k"], a["C0"], a["it"], a["tol"], a["a"],
                                  a["c"], None, 0, C.byref(st))

    assert call(it=0) == N.KM_ERR_INVALID_ARG
    assert call(tol=-1.0) == N.KM_ERR_INVALID_ARG
    assert call(tol=math.nan) == N.KM_ERR_INVALID_ARG
    assert call(a=None) == N.KM_ERR_INVALID_ARG
    assert call(c=None) == N.KM_ERR_INVALID_ARG
    assert call(k=11) == N.KM_ERR_INVALID_ARG
    assert call(X=None) == N.KM_ERR_INVALID_ARG


def test_pp_seed_rejects_bad_arguments_without_a_device():
    lib = N.load()
    fake = C.c_void_p(0x1000)
    need = lib.kmeans_pp_workspace_bytes(10, 2, 3)
    assert need > 10 * 12
    assert lib.kmeans_pp_workspace_bytes(10, 2, 11) == 0
    assert lib.kmeans_pp_workspace_bytes(0, 2, 1) == 0
    good = dict(X=fake, n=10, d=2, k=3, u=[0.1, 0.5, 0.9], C=fake, ws=fake, wsb=need, flags=0)

    def call(**kw):
        a = dict(good, **kw)
        u = (C.c_double * len(a["u"]))(*a["u"])
        return lib.kmeans_pp_seed(a["X"], a["n"], a["d"], a["k"], u, a["C"], None, None, a["ws"], a["wsb"],
                                  a["flags"], None, None)

    assert call(k=11, u=[0.5] * 11) == N.KM_ERR_INVALID_ARG
    assert call(k=0, u=[0.5]) == N.KM_ERR_INVALID_ARG
    assert call(X=None) == N.KM_ERR_INVALID_ARG
    assert call(C=None) == N.KM_ERR_INVALID_ARG
    assert call(u=[0.1, 1.0, 0.2]) == N.KM_ERR_INVALID_ARG
    assert call(u=[0.1, -0.5, 0.2]) == N.KM_ERR_INVALID_ARG
    assert call(u=[0.1, math.nan, 0.2]) == N.KM_ERR_INVALID_ARG
    assert call(flags=4) == N.KM_ERR_INVALID_ARG
    assert call(wsb=need - 1) == N.KM_ERR_INVALID_ARG
    assert call(ws=C.c_void_p(0x1008)) == N.KM_ERR_INVALID_ARG


def test_null_context_calls():
    lib = N.load()
    ch = C.c_int64(0)
    st = N.KmStats()
    assert lib.kmeans_mti_iterate(None, C.byref(ch)) == N.KM_ERR_INVALID_ARG
    assert lib.kmeans_mti_get(None, None, None) == N.KM_ERR_INVALID_ARG
    assert lib.kmeans_mti_get_centroids64(None, None) == N.KM_ERR_INVALID_ARG
    assert lib.kmeans_mti_get_stats(None, C.byref(st)) == N.KM_ERR_INVALID_ARG
    assert lib.kmeans_mti_get_history(None, None, None, None, None, None, 4) == N.KM_ERR_INVALID_ARG
    lib.kmeans_mti_destroy(None)   # NULL-safe


def test_binding_rejects_cpu_tensors():
    import torch
    import paper_1902_09527_amd as km
    X = torch.zeros(10, 2)
    with pytest.raises(ValueError):
        km.run(X, X[:2].clone(), 5)
    with pytest.raises(ValueError):
        km.KMeansMTI(X, X[:2].clone())
