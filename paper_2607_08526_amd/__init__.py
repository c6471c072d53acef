"""Block-quantized (int8 / q4, block 32, fp16 scale) linear layers for MI355X.

The library is libqlinear.so (C ABI in include/qlinear.h, HIP kernels for
gfx950 in csrc/); `qlinear` is its Python binding.
"""
__all__ = ["qlinear", "build"]
