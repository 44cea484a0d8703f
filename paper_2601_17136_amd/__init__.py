"""MI355X-native exact Kernel K-means engine (arxiv 2601.17136, single GPU).

The engine is the C-ABI shared library ``libkkm.so`` built from ``csrc/``
(hand-written HIP kernels for gfx950 plus a C++ host layer).  ``kkm`` is the
thin ctypes binding to it; ``datagen`` draws the seeded synthetic workloads.
Importing this package loads nothing: the library is opened on first use and
a missing library is an error, never a fallback.
"""

__all__ = ["kkm", "datagen"]
