"""Urgency-Aware Denoising (UAD) action-expert hot path for AMD MI355X (gfx950).

The compute runs in ``libuad.so`` (hand-written HIP kernels behind the C ABI
of ``include/uad.h``); this package is its thin Python binding plus a small
convenience wrapper, :class:`ActionExpert`, used by the tests and the benchmark.
"""
from ._binding import *  # noqa: F401,F403
from ._binding import __all__ as _b_all
from .expert import ActionExpert

__all__ = list(_b_all) + ["ActionExpert"]
