"""MI355X (gfx950) structured sketches (FJL, FFD, AFFD, AFJL, QK and the Q-pre-conditioned kinds) and
the sketched HVP operator with Arnoldi in the sketched space, behind a C ABI.

The kernels live in libsketch.so (csrc/, built by build.py); this package only
marshals torch tensors into that library.
"""
from .sketch import KINDS, Sketch  # noqa: F401
from ._lib import SketchError  # noqa: F401
from .hvp import SyntheticHessian, arnoldi, arnoldi_step, id_search, ritz_values, sketch_hvp  # noqa: F401
