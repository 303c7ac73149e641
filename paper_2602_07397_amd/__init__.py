"""MI355X (gfx950) Sketch&Walk sparse-attention hot path.

The computation lives in libsketchwalk.so (HIP kernels behind a C ABI, see
include/sketchwalk.h); :mod:`.binding` is a thin ctypes layer over it.
"""
from . import binding  # noqa: F401
from .binding import SketchWalkError  # noqa: F401

__all__ = ["binding", "SketchWalkError"]
