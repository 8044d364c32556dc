"""MI355X-native LouisKV KV clustering and retrieval path.

The compute lives in libLouisKV (HIP for gfx950, C ABI in include/louiskv.h);
this package is its binding (`louiskv`), an engine that owns a batch's
buffers and issues the calls in the paper's Algorithm 1 order (`engine`), and
the build step (`build`).
"""
from . import louiskv
from .louiskv import LouisKVError, load_library

__all__ = ["louiskv", "LouisKVError", "load_library"]
