"""MI355X (gfx950) implementation of DynaSpec's dynamic draft head.

The work runs in libdynahead.so (hand-written HIP kernels behind a C ABI,
declared in include/dynahead.h); `dynahead` is its Python binding.
"""
from . import dynahead  # noqa: F401

__all__ = ["dynahead"]
