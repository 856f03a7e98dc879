"""MI355X-native tree-packed chunkwise linear attention (HARTS, arXiv 2608.28158).

The compute path is libharts.so (include/harts.h): a host planner and HIP
kernels for gfx950.  This package is its thin Python binding.
"""
from . import _lib  # noqa: F401

__all__ = ["plan", "tree_la"]
