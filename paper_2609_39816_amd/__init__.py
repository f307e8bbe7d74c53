"""MI355X-native FP8 evaluation of bilinear fast matrix multiplication
schemes across gauge orbits (Xie et al., "Beyond Accuracy: Prefix-Invariant
Realizations of Low-Precision Fast Matrix Multiplication").

The compute lives in libfm (HIP kernels for gfx950 behind the C ABI of
include/fm.h); `paper_2609_39816_amd.fm` is its Python binding.
"""
from . import schemes  # noqa: F401
