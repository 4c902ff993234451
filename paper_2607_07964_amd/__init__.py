"""KronQ per-layer quantisation path for AMD MI355X (gfx950).

``kronq`` is the ctypes binding of libkronq.so (HIP kernels behind a C ABI, include/kronq.h);
``layer`` chains its calls into the per-layer hot path. Build the library with
``python -m paper_2607_07964_amd.build``.
"""
from . import kronq  # noqa: F401
from .kronq import KronqError, load  # noqa: F401

__all__ = ["kronq", "layer", "load", "KronqError"]
