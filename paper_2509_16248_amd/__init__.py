"""MI355X-native graph-break-free transformer forward (libgm).

``gm``    -- ctypes binding of include/gm.h (same names as the C ABI)
``model`` -- GmModel: torch-facing wrapper (device memory and streams)
``build`` -- compiles libgm.so for gfx950
"""
from . import gm  # noqa: F401
