"""MI355X-native hot path of risk-aware overlapping-subgraph GNN training.

The compute path lives in ``libhg.so`` (hand-written HIP kernels for gfx950
behind a C ABI, declared in ``include/hg.h``).  ``api`` is a thin ctypes
binding with the same entry-point names; ``synth`` draws seeded synthetic
inputs.  Importing this package loads nothing: ``api`` loads the library on
first use and raises if it has not been built.
"""
__all__ = ["api", "synth"]
