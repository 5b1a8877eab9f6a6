"""MI355X (gfx950) implementation of the Jorge optimizer step.

The step runs in hand-written HIP kernels behind the C ABI of include/jorge.h
(libjorge.so, built in-tree by paper_2310_12298_amd.build). This package holds
that library's sources, its ctypes binding and the seeded synthetic workloads.
Importing it does not load the library; constructing Jorge does, and raises
if the library is missing.
"""
__all__ = ["Jorge", "JorgeError", "load_library"]


def __getattr__(name):
    if name in __all__:
        from . import jorge
        return getattr(jorge, name)
    raise AttributeError(name)
