"""wsr: weight-streaming read kernels for MI355X (gfx950).

The product is libwsr.so (include/wsr.h); `paper_2608_12114_amd.wsr` is its Python binding.
"""
from . import wsr  # noqa: F401  (fails loudly if libwsr.so is not built)
from .wsr import *  # noqa: F401,F403
