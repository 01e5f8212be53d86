"""MI355X-native merged multi-model CNN inference (GEMEL model merging,
arXiv 2201.07705): libgemel.so (HIP kernels for gfx950 behind a C ABI,
include/gemel.h) and its ctypes binding."""

from .gemel import Context, GemelError, lib  # noqa: F401
