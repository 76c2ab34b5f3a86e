"""Carry-through checksum CNN inference on MI355X (gfx950).

``ctc`` is the ctypes binding of libctc.so (include/ctc.h); ``CtcNet`` owns
a bound network.  Importing fails if the HIP library is not built.
"""
from . import ctc  # noqa: F401
from .runtime import CtcNet  # noqa: F401
