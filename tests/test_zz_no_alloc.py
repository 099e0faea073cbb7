"""kmeans_pp_seed_noalloc (static device workspace, no allocation) against
kmeans_pp_seed (caller's workspace), through the C ABI.

Seeding is index work decided by float64 arithmetic, so the bar is
bit-exact: the same seed indices, seed rows and D2 values.  Two calls in a
row, the second on a smaller input, so the second sees the first call's
contents left in the shared array.
"""
import ctypes as C

import numpy as np
import pytest
import torch

import synth
from paper_1902_09527_amd import _native as N

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _seed(lib, fn, X, k, u, prune, ws=None):
    n, d = X.shape
    c = torch.full((k, d), -1.0, dtype=torch.float32, device=DEV)
    idx = torch.full((k,), -1, dtype=torch.int64, device=DEV)
    d2 = torch.full((n,), -1.0, dtype=torch.float64, device=DEV)
    uu = np.ascontiguousarray(u, np.float64)
    flags = 0 if prune else N.KM_PP_NO_PRUNE
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    P = C.c_void_p
    if ws is None:
        st = lib.kmeans_pp_seed_noalloc(P(X.data_ptr()), n, d, k, uu.ctypes.data_as(P), P(c.data_ptr()),
                                        P(idx.data_ptr()), P(d2.data_ptr()), flags, stream)
    else:
        st = lib.kmeans_pp_seed(P(X.data_ptr()), n, d, k, uu.ctypes.data_as(P), P(c.data_ptr()),
                                P(idx.data_ptr()), P(d2.data_ptr()), P(ws.data_ptr()), ws.numel(), flags,
                                stream, None)
    assert st == N.KM_OK, (fn, st, lib.kmeans_mti_last_hip_error())
    torch.cuda.synchronize()
    return idx.cpu().numpy(), c.cpu().numpy(), d2.cpu().numpy()


@pytest.mark.parametrize("prune", [True, False], ids=["prune", "noprune"])
def test_noalloc_matches_workspace_entry_point_twice(prune):
    lib = N.load()
    cases = [(401, 300000 + 7, 32, 20), (402, 50000 + 3, 16, 9)]   # second call smaller
    for seed, n, d, k in cases:
        print("case", seed, n, d, k, prune, flush=True)
        X, _ = synth.blobs(n, d, max(k // 2, 1), seed=seed, spread=4.0, sigma=1.0)
        Xg = torch.from_numpy(X).to(DEV)
        u = np.random.default_rng(seed).random(k)
        need = int(lib.kmeans_pp_workspace_bytes(n, d, k))
        assert 0 < need <= N.KMEANS_PP_STATIC_WORKSPACE_BYTES
        ws = torch.empty(need, dtype=torch.uint8, device=DEV)   # the caching allocator aligns to 512 B
        assert ws.data_ptr() % 256 == 0
        want = _seed(lib, "kmeans_pp_seed", Xg, k, u, prune, ws)
        got = _seed(lib, "kmeans_pp_seed_noalloc", Xg, k, u, prune)
        np.testing.assert_array_equal(got[0], want[0])
        np.testing.assert_array_equal(got[1], want[1])
        np.testing.assert_array_equal(got[2], want[2])
        np.testing.assert_array_equal(got[1], X[want[0]])


def test_noalloc_refuses_sizes_beyond_the_static_workspace():
    lib = N.load()
    X, _ = synth.blobs(4096, 8, 4, seed=403)
    Xg = torch.from_numpy(X).to(DEV)
    c = torch.empty(4, 8, dtype=torch.float32, device=DEV)
    u = np.full(4, 0.5)
    P = C.c_void_p
    big_n = 10_000_000   # needs about 120 MB of workspace; refused before any pointer is read
    assert lib.kmeans_pp_workspace_bytes(big_n, 8, 4) > N.KMEANS_PP_STATIC_WORKSPACE_BYTES
    st = lib.kmeans_pp_seed_noalloc(P(Xg.data_ptr()), big_n, 8, 4, u.ctypes.data_as(P), P(c.data_ptr()),
                                    None, None, 0, None)
    assert st == N.KM_ERR_INVALID_ARG
    assert b"static workspace" in lib.kmeans_mti_last_hip_error()
    st = lib.kmeans_pp_seed_noalloc(P(Xg.data_ptr()), 4096, 8, 4, u.ctypes.data_as(P), P(c.data_ptr()),
                                    None, None, N.KM_PP_TIMING, None)
    assert st == N.KM_ERR_INVALID_ARG
