"""REAL-Q per-layer quantization sweep on MI355X (gfx950).

The compute lives in librealq.so (C ABI in include/realq.h); ``paper_2609_00049_amd.realq``
is its Python binding and raises ImportError when the library has not been built
(``paper_2609_00049_amd.build.build()``).
"""
__all__ = ["realq", "build"]
