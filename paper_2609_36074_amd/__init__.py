"""MI355X (gfx950) NLR K-means iteration: C-ABI library libnlr.so + thin binding.

The product path is ``paper_2609_36074_amd.nlr`` over ``libnlr.so`` (built
from ``csrc/`` by ``_build.py``).  It never imports the test oracle.
"""
from . import nlr  # noqa: F401

__all__ = ["nlr"]
