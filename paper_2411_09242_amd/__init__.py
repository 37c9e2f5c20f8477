"""MI355X-native hot path of FluidML (arXiv 2411.09242): layout-planned,
arena-planned transformer operator chain on hand-written HIP kernels.

The native library (lib/libfluid.so, built by ``paper_2411_09242_amd.build``)
does all the work; ``paper_2411_09242_amd.fluid`` is its ctypes binding.
"""
from . import fluid  # noqa: F401
from .fluid import load  # noqa: F401
