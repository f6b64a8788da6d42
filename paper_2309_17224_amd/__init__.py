"""FP8 linear layer with per-tensor power-of-two scaling biases on MI355X.

The compute path is libfp8lin.so (hand-written HIP for gfx950, C ABI in
include/fp8lin.h); ``paper_2309_17224_amd.fp8lin`` is its ctypes binding and
``paper_2309_17224_amd.linear`` chains the calls into the training and
inference steps of the method.  Importing the package loads nothing.
"""
__all__ = ["fp8lin", "linear", "workloads", "build"]
