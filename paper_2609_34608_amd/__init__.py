"""MI355X (gfx950) hot path of training-free World Action Model inference.

The compute lives in ``lib/libwam.so`` (HIP kernels behind a C ABI declared
in ``include/wam.h``); ``runtime.WamModel`` is its Python binding.
"""
from . import _lib  # noqa: F401

__all__ = ["runtime", "_lib"]
