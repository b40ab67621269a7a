"""MI355X-native hashed shared-memory embedding layer (PSS / ROBE-Z).

libpss.so (HIP, gfx950) does all the work; ``pss`` is its ctypes binding.
"""
from . import pss  # noqa: F401
