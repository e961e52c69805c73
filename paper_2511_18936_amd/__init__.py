"""SWAN decode attention on a rotated-and-pruned KV cache, for MI355X (gfx950).

The compute path lives in libswan.so (HIP kernels behind the C ABI of
include/swan.h); ``swan`` is its ctypes binding.
"""
from . import swan  # noqa: F401
from .swan import (CacheDesc, SwanCache, SwanError, calibrate_rotation,  # noqa: F401
                   compress_append, decode_attention)
