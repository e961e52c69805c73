"""SWAN decode attention on a rotated-and-pruned KV cache, for MI355X (gfx950).

The compute path lives in libswan.so (HIP kernels behind the C ABI of
include/swan.h); ``swan`` is its ctypes binding, loaded on first use so that
``paper_2511_18936_amd.build`` can run before the library exists.
"""
import importlib

__all__ = ["swan", "build"]


def __getattr__(name):
    if name in ("swan", "build"):
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
