"""Adaptive dynamic-shape GEMM for MI355X (gfx950).

Python binding of the C ABI in include/adaptcore.h. The computation runs in
the HIP kernels of libadaptcore.so; this package only marshals arguments.
"""
from ._lib import *  # noqa: F401,F403
from ._lib import lib, last_error, AdaptCoreError, matmul_tensors, addmm_tensors, bmm_tensors, grouped_mm_tensors  # noqa: F401,E501
