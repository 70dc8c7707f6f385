"""SPLA decode step on AMD Instinct MI355X (gfx950).

The product is libspla.so, a C-ABI library of hand-written HIP kernels
(include/spla.h); `paper_2601_22379_amd.spla` is its Python binding.
"""

from . import spla  # noqa: F401

__all__ = ["spla"]
