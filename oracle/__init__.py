"""fp64 CPU oracle for the NLR K-means iteration — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import anything from this package.  The product path (the
HIP library and its Python binding) never does, and shares no code with it.

Modules:
  nlr     plain unfused Algorithm 1 in float64 (factored form, never forms Ahat)
  dense   explicit n x n cross-form of the same step (small n only)
  kmeans  brute-force exact K-means by partition enumeration, ARI, CNR threshold
"""
from . import dense, kmeans, nlr

__all__ = ["nlr", "dense", "kmeans"]
