"""MI355X-native compression hot path of SDP4Bit (arXiv 2410.15526).

The work happens in ``libsdp4.so`` (hand-written HIP kernels for gfx950
behind the C ABI of ``include/sdp4.h``); :mod:`paper_2410_15526_amd.sdp4`
is a thin ctypes binding with the same names.  Importing this package does
not load the library; the first call does, and raises if it is missing.
"""
from . import sdp4  # noqa: F401

__all__ = ["sdp4"]
