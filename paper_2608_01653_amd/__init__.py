"""MI355X-native Hadamard-domain INT8 linear operator (HaTQ inference hot path).

``hatq``      -- ctypes binding of libhatq.so (C ABI in include/hatq.h)
``synth``     -- seeded synthetic inputs (no method arithmetic)
``workloads`` -- the layer shapes and input recipes
``build``     -- hipcc build of libhatq.so for gfx950
"""
from . import synth, workloads  # noqa: F401

__all__ = ["synth", "workloads"]
