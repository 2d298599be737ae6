"""MI355X-native DP-SGD gradient-step hot path (Opacus, arXiv 2109.12298).

The product is ``libdpgrad.so``, a C-ABI library of hand-written HIP kernels
for gfx950 (declared in ``include/dpgrad.h``).  ``binding`` is a thin ctypes
layer over it with the same entry-point names; ``step`` strings the calls of
one DP-SGD step together; ``workloads`` draws seeded synthetic inputs.
Nothing is loaded at import time.
"""
__all__ = ["binding", "step", "workloads", "build"]
