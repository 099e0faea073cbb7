"""MI355X-native hot path of clusterNOR's k-means (arXiv 1902.09527).

Lloyd's k-means with Minimal Triangle Inequality pruning as hand-written HIP
kernels for gfx950 behind a C ABI (include/kmeans_mti.h); this package holds
the kernels (csrc/), the build step (build.py) and a thin ctypes binding.
"""
from .kmeans import KMeansMTI, kmeanspp, kmeanspp_workspace_bytes, run, run_pp_best  # noqa: F401

__all__ = ["KMeansMTI", "kmeanspp", "kmeanspp_workspace_bytes", "run", "run_pp_best"]
