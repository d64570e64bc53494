"""MI355X (gfx950) implementation of the COUNTDOWN sparse Gated-MLP FFN.

The hot path lives in ``libcountdown.so`` (HIP kernels + C ABI, declared in
``include/countdown.h``); :mod:`.binding` is its thin ctypes front end and
:mod:`.traffic` counts the algorithmic bytes and FLOPs the kernels must move.
Importing the package loads nothing; the library is loaded on first use.
"""
from . import traffic  # noqa: F401

__all__ = ["binding", "traffic", "build"]
