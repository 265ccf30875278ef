"""MI355X-native microscaled-FP4 attention forward (SageAttention3, arXiv 2505.11594).

The compute path is a C-ABI shared library of hand-written HIP kernels for
gfx950 (``csrc/``, declared in ``include/sage_mi355x.h``); ``binding`` is a
thin ctypes layer over it.  ``workloads`` holds the seeded input generators.
"""
