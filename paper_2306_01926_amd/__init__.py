"""MI355X-native group attention (RITA, arXiv 2306.01926).

The computation lives in libga.so (HIP kernels for gfx950 behind the C ABI of
include/ga.h); `ga` is its Python binding and `inputs` the seeded synthetic
input generator.
"""
from . import ga, inputs  # noqa: F401

__all__ = ["ga", "inputs"]
