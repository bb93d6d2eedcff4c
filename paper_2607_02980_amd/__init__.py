"""MI355X-native HiLS (Hierarchical Landmark Sparse) attention.

The operator lives in ``libhils.so`` (hand-written HIP for gfx950) behind the
C-ABI declared in ``include/hils.h``; ``paper_2607_02980_amd.hils`` is the thin
ctypes binding with the same entry-point names.
"""
