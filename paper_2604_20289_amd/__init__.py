"""MI355X (gfx950) X-Cache cached chunk forward: HIP kernels behind a C ABI.

``xcache`` is the ctypes binding of ``libxcache.so``; ``build`` compiles it.
"""
from . import xcache  # noqa: F401
from .xcache import XCache, load_library  # noqa: F401
