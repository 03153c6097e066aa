"""MI355X-native Zipf gradient compression (Unique -> Seg-Sum -> Fill-Values)
from "Language Modeling at Scale" (arXiv:1810.10045).

The compute lives in ``liblmzipf.so`` (hand-written HIP for gfx950, C ABI in
``include/lmzipf.h``); ``paper_1810_10045_amd.lmzipf`` is the thin ctypes
binding with the same entry-point names. Importing this package does not load
the library; the binding does, and raises if it is missing.
"""
import importlib

__all__ = ["lmzipf", "synth"]


def __getattr__(name):
    if name in __all__:
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
