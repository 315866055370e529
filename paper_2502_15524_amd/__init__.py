"""MI355X pipeline-stage engine for cold-start LLM serving.

The engine is libhs.so (C ABI in include/hs.h, HIP kernels for gfx950);
``hs`` is its ctypes binding and ``pipeline`` holds marshalling helpers.
"""
from . import hs  # noqa: F401

__all__ = ["hs"]
