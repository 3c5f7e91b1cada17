"""Layer-parallel training of deep residual networks (arXiv:1812.04352) on MI355X.

The hot path (layer-serial and MGRIT/FAS forward and adjoint solves, the reduced
gradient and the residual norm) lives in the HIP library liblp.so behind the C
ABI of include/lp.h; ``paper_1812_04352_amd.lp`` is its thin Python binding.
"""
from . import lp  # noqa: F401

__all__ = ["lp"]
