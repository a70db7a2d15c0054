"""MI355X (gfx950) GCN training hot path: Morphling's fused aggregation with the
sparsity-aware dense/sparse switch (arXiv 2512.01678), as a C-ABI HIP library
(libgcn.so, declared in include/gcn.h) with a thin ctypes binding (gcn.py).
"""
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgcn.so")


def build(verbose: bool = False) -> str:
    """Compile libgcn.so for gfx950 (hipcc)."""
    from . import _build
    return _build.build(verbose=verbose)
