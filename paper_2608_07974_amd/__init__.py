"""ZeroLock chunk-local update on MI355X (gfx950).

libzl (HIP kernels + C ABI, include/zl.h) computes the whole update; zl.py is
its ctypes binding and chunk.py keeps the buffers in torch device tensors.
"""
from . import zl  # noqa: F401

__all__ = ["zl"]
