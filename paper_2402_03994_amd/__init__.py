"""MI355X (gfx950) structured sketches: FJL, FFD, AFFD, AFJL and QK behind a C ABI.

The kernels live in libsketch.so (csrc/, built by build.py); this package only
marshals torch tensors into that library.
"""
from .sketch import KINDS, Sketch  # noqa: F401
from ._lib import SketchError  # noqa: F401
