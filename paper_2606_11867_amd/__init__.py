"""ForeMoE per-micro-step MoE expert layer on MI355X (gfx950).

The compute lives in libforemoe.so (hand-written HIP kernels behind the C ABI
of include/foremoe.h); this package is its thin binding. Importing it does
not touch the GPU; ``load()`` loads the library and raises if it is missing.
"""
from ._lib import load, ForeMoEError, LIB_PATH  # noqa: F401

__all__ = ["load", "ForeMoEError", "LIB_PATH"]
