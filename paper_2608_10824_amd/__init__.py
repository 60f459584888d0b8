"""Gated VLA-Cache control step on MI355X (gfx950).

libgvc.so (C ABI in include/gvc.h) holds the whole hot path as HIP kernels;
`gvc` is its ctypes binding and `session.Session` a PyTorch-allocated
wrapper around one context.
"""
from . import gvc

__all__ = ["gvc"]
