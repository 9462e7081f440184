"""OmniTide's per-chunk stream step on AMD Instinct MI355X (gfx950).

The product is ``libomnitide.so`` (hand-written HIP kernels behind the C ABI declared in
``include/omnitide.h``).  ``omnitide`` is its thin ctypes binding (same function names) and
``step.StreamStep`` drives one score -> select -> compact -> attend step on a HIP stream.
"""
from . import omnitide  # noqa: F401
from .omnitide import OmnitideError, lib, version  # noqa: F401

__all__ = ["omnitide", "OmnitideError", "lib", "version"]
