"""Cache-aware MoE decode step on MI355X (gfx950): native HIP kernels behind a
C ABI (include/cmoe.h), with a thin ctypes binding in ``cmoe``.

Importing the package does not load the library; ``cmoe.lib()`` does, and
raises if libcmoe.so has not been built.  There is no CPU fallback.
"""
from . import cmoe  # noqa: F401
from .cmoe import CmoeError, Engine, cmoe_query, lib, make_config  # noqa: F401
