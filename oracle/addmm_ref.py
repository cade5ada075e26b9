"""AddMM oracle -- TEST INFRASTRUCTURE ONLY.

Only tests, the smoke check and the benchmark's CPU-baseline leg may import
this module; it shares no code with the GPU library.

AddMM is one of the dense operators the paper replaces in its end-to-end
models next to MatMul (Section 6.5; operator scope, Section 7). The paper
names the operator but does not write it out; it is read here with its usual
meaning, a scaled product plus a scaled input plus a bias row broadcast over
the rows:

    C[i][j] = alpha * sum_k A[i][k] * B[k][j] + beta * C_old[i][j] + bias[j]

with the product taken from the plain-product oracle (gemm_ref) in fp64.
When beta == 0 the input C_old takes no part at all (it may hold NaN or
garbage, as with the BLAS convention); bias None means no bias term.

The acceptance scale of an entry is the sum of the magnitudes of its terms,

    D[i][j] = |alpha| * sum_k |A[i][k] B[k][j]| + |beta| |C_old[i][j]| + |bias[j]|,

so that the GPU's fp32 epilogue rounding and the final rounding to a 16-bit
output are measured against the same relative bars as a plain product.

The batched form (BatchMM with the same epilogue) applies it to every batch
of the strided batched product (grouped_ref.batched_gemm), with one bias row
shared by all batches; the grouped form (GroupMM with the same epilogue)
applies it to the covered rows of the grouped product (grouped_ref), group g
adding its own bias row, stored stride_bias values after group g-1's.

Parity pins: tests/test_oracle_addmm.py (exact rational brute force of C and
D on tiny inputs with mixed-sign alpha and beta, reduction to the plain
product, beta == 0 ignoring a NaN C_old, K == 0, sampled entries equal to
the full result, every batch of the batched form equal to the single form on
that batch's matrices, every group of the grouped form equal to the single
form on that group's rows and bias row, and a mutation test).
"""
import numpy as np

from . import gemm_ref
from . import grouped_ref


def addmm(A, B, C_old, alpha, beta, bias=None, M=None, N=None, K=None, lda=None, ldb=None, fmt="bf16",
          lib=None):
    """(C_ref, D) of AddMM in fp64, both M x N.

    A, B: uint16 bit patterns as for gemm_ref.gemm; C_old: M x N values (the
    previous content of C, already decoded to numbers); bias: N values or
    None.
    """
    P, Dp = gemm_ref.gemm(A, B, M=M, N=N, K=K, lda=lda, ldb=ldb, fmt=fmt, lib=lib)
    alpha = float(alpha)
    beta = float(beta)
    C = alpha * P
    D = abs(alpha) * Dp
    if beta != 0.0:
        Co = np.asarray(C_old, np.float64).reshape(C.shape)
        C = C + beta * Co
        D = D + abs(beta) * np.abs(Co)
    if bias is not None:
        b = np.asarray(bias, np.float64).reshape(1, C.shape[1])
        C = C + b
        D = D + np.abs(b)
    return C, D


def addmm_entries(A, B, I, J, c_old, alpha, beta, bias, M=None, N=None, K=None, lda=None, ldb=None, fmt="bf16",
                  lib=None):
    """Entries (I[t], J[t]) of AddMM, each from its A row and B column (the
    plain oracle's gemm_entries); c_old[t] is C_old at that entry and
    bias[t] the bias of its column (None: no bias)."""
    P, Dp = gemm_ref.gemm_entries(A, B, I, J, M=M, N=N, K=K, lda=lda, ldb=ldb, fmt=fmt, lib=lib)
    alpha = float(alpha)
    beta = float(beta)
    C = alpha * P
    D = abs(alpha) * Dp
    if beta != 0.0:
        Co = np.asarray(c_old, np.float64).reshape(C.shape)
        C = C + beta * Co
        D = D + abs(beta) * np.abs(Co)
    if bias is not None:
        b = np.asarray(bias, np.float64).reshape(C.shape)
        C = C + b
        D = D + np.abs(b)
    return C, D


def batched_addmm(A, B, C_old, batch, M, N, K, lda, ldb, stride_a, stride_b, alpha, beta, bias=None, fmt="bf16",
                  lib=None):
    """(C_ref, D) of shape (batch, M, N): the epilogue above applied to every
    batch of the strided batched product; C_old has shape (batch, M, N)."""
    P, Dp = grouped_ref.batched_gemm(A, B, batch, M, N, K, lda, ldb, stride_a, stride_b, fmt=fmt, lib=lib)
    alpha = float(alpha)
    beta = float(beta)
    C = alpha * P
    D = abs(alpha) * Dp
    if beta != 0.0:
        Co = np.asarray(C_old, np.float64).reshape(C.shape)
        C = C + beta * Co
        D = D + abs(beta) * np.abs(Co)
    if bias is not None:
        b = np.asarray(bias, np.float64).reshape(1, 1, N)
        C = C + b
        D = D + np.abs(b)
    return C, D


def grouped_addmm(A, B, counts, rows, N, K, lda, ldb, stride_b, C_old, alpha, beta, bias=None, stride_bias=0,
                  fmt="bf16", lib=None):
    """(C_ref, D, covered) of the grouped form, C_ref and D of shape (rows, N)
    (uncovered rows 0); C_old has shape (rows, N); bias is a flat array with
    group g's row at g * stride_bias."""
    P, Dp, covered = grouped_ref.grouped_gemm(A, B, counts, rows, N, K, lda, ldb, stride_b, fmt=fmt, lib=lib)
    alpha = float(alpha)
    beta = float(beta)
    C = alpha * P
    D = abs(alpha) * Dp
    if beta != 0.0:
        Co = np.where(covered[:, None], np.asarray(C_old, np.float64).reshape(rows, N), 0.0)
        C = C + beta * Co
        D = D + abs(beta) * np.abs(Co)
    if bias is not None:
        bias = np.asarray(bias, np.float64).reshape(-1)
        for g, (s, e) in enumerate(grouped_ref.group_rows(counts, rows)):
            if e > s:
                b = bias[g * stride_bias:g * stride_bias + N].reshape(1, N)
                C[s:e] = C[s:e] + b
                D[s:e] = D[s:e] + np.abs(b)
    return C, D, covered
