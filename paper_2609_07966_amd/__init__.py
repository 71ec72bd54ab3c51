"""MI355X-native decode attention over MetaKV's KV-cache compression configurations.

libmkv.so (HIP kernels for gfx950 behind the C ABI in include/mkv.h) does the work; ``_lib`` binds
it with ctypes and ``cache.KVCache`` marshals torch tensors to it.
"""
from . import _lib  # noqa: F401
