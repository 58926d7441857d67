"""EchoCache cached DiT block step on MI355X (gfx950).

The compute path is libecho.so (HIP kernels behind the C ABI in
include/echo.h); this package only loads it and marshals torch tensors.
"""
from . import _lib  # noqa: F401
from ._lib import EchoError, load  # noqa: F401

__version__ = "0.1.0"

