"""MI355X-native conv2d hot path for DML-style deep learning (gfx950, HIP).

The compute lives in ``libdmlnn.so`` (hand-written HIP kernels behind a C ABI,
declared in ``include/dmlnn.h``).  ``paper_1802_04647_amd.dmlnn`` is the thin
Python binding; importing this package loads nothing, and the first call into
the binding fails loudly if the library is missing.
"""
__all__ = ["dmlnn", "inputs"]
