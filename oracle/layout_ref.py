"""Operand layouts of the plain product -- TEST INFRASTRUCTURE ONLY.

Only tests, the smoke check and the benchmark's CPU-baseline leg may import
this module; it shares no code with the GPU library.

The paper's padding module copies operands whose layout the main kernel
cannot read efficiently into an aligned form in a prologue (Table 2;
Section 5, the T_pro term of Eq. 7). The product itself does not depend on
how an operand is stored: with A stored column-major, element (i, k) of A is
the stored element at i + k * lda; with B stored column-major, element (k, j)
of B is at k + j * ldb; row-major storage puts them at i * lda + k and
k * ldb + j. This module reads the logical matrices out of the stored arrays
by exactly those index rules (a strided view, then a contiguous copy) and
hands them to the plain-product oracle.

Parity pins: tests/test_oracle_layouts.py (exact rational brute force that
indexes the stored arrays by the rules above, for all four layouts with
padded leading dimensions; a column-major operand stored as the row-major
transpose gives the row-major product bit for bit; mutations of the index
rules each fail a pin).
"""
import numpy as np

from . import gemm_ref

A_COL = 1
B_COL = 2


def logical(mem, rows, cols, ld, col_major):
    """The rows x cols matrix stored in the flat uint16 array `mem`, as a
    contiguous row-major array."""
    mem = np.ascontiguousarray(mem).reshape(-1)
    if rows == 0 or cols == 0:
        return np.zeros((rows, cols), np.uint16)
    if col_major:
        last, strides = (rows - 1) + (cols - 1) * ld, (2, 2 * ld)
    else:
        last, strides = (rows - 1) * ld + (cols - 1), (2 * ld, 2)
    if last >= mem.size:
        raise ValueError("the stored array is too short for its shape and leading dimension")
    view = np.lib.stride_tricks.as_strided(mem, shape=(rows, cols), strides=strides)
    return np.ascontiguousarray(view)


def gemm_layout(A_mem, B_mem, M, N, K, lda, ldb, layouts, fmt="bf16", lib=None):
    """(C_ref, D) of C = A * B with A and B read from their stored arrays
    under `layouts` (bit A_COL: A column-major, bit B_COL: B column-major)."""
    A = logical(A_mem, M, K, lda, bool(layouts & A_COL))
    B = logical(B_mem, K, N, ldb, bool(layouts & B_COL))
    return gemm_ref.gemm(A, B, M=M, N=N, K=K, fmt=fmt, lib=lib)
