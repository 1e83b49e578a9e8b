"""LM-GC on MI355X: the data-parallel hot path of "Language Models as Zero-shot
Lossless Gradient Compressors" (arXiv 2409.17836) as hand-written HIP for
gfx950 behind the C ABI of include/lmgc.h (liblmgc.so).

`binding` is the ctypes layer (argument marshalling only); `_build` compiles
the library in-tree.
"""
from . import binding  # noqa: F401

__all__ = ["binding"]
