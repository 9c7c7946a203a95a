"""Spreeze's large-batch actor-critic update on one MI355X (gfx950).

The update runs in libspz.so (hand-written HIP behind the C ABI of
include/spz.h); `spz` is its ctypes binding and `build` compiles it.
"""
from .spz import Spz, SpzError, load  # noqa: F401
