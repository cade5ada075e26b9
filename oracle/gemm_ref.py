"""Python side of the GEMM oracle (test infrastructure only).

Only tests, the smoke check and the benchmark's CPU-baseline leg may import
this module. It loads the oracle's own C library (gemm_ref.c) and shares no
code with the GPU library.

What it provides:
  * gemm(A, B, ...)          -> (C_ref, D) in fp64, rows [row0, row1)
  * gemm_entries(A, B, I, J) -> single entries, for checks at full size
  * decode(bits, fmt)        -> fp64 values of bf16 / fp16 bit patterns
  * err_metric(C, C_ref, D)  -> max_ij |C - C_ref| / D_ij, the acceptance
                                measure for the GPU results. Where D_ij is 0
                                (a zero row of A or column of B) the entry
                                must be exactly 0, otherwise the metric is inf.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgemm_ref.so")

FMT = {"bf16": 0, "fp16": 1}

_lib = None


def load(path=None):
    """Load (building if needed) the oracle library. `path` is for tests."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(LIB_PATH) or (
                os.path.getmtime(LIB_PATH) < os.path.getmtime(os.path.join(HERE, "gemm_ref.c"))):
            from . import build as _b
            _b.build()
        _lib = _bind(ctypes.CDLL(LIB_PATH))
    return _lib


def _bind(lib):
    i64, p = ctypes.c_int64, ctypes.c_void_p
    lib.oracle_gemm.argtypes = [ctypes.c_int, i64, i64, i64, p, i64, p, i64, p, p, i64, i64, i64]
    lib.oracle_gemm.restype = ctypes.c_int
    lib.oracle_gemm_entries.argtypes = [ctypes.c_int, i64, i64, i64, p, i64, p, i64, p, p, i64, p, p]
    lib.oracle_gemm_entries.restype = ctypes.c_int
    lib.oracle_decode.argtypes = [ctypes.c_int, p, p, i64]
    lib.oracle_decode.restype = None
    lib.oracle_threads.argtypes = []
    lib.oracle_threads.restype = ctypes.c_int
    return lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _as_u16(x):
    x = np.asarray(x)
    if x.dtype != np.uint16:
        raise TypeError("oracle inputs are 16-bit bit patterns (uint16), got %s" % x.dtype)
    return x


def gemm(A, B, M=None, N=None, K=None, lda=None, ldb=None, fmt="bf16",
         rows=None, want_d=True, lib=None):
    """C_ref = A @ B in fp64 from bf16/fp16 bit patterns.

    A and B are 2-D uint16 arrays (row-major, possibly with padded rows: pass
    M, N, K and lda, ldb to use a sub-matrix). `rows` = (row0, row1) restricts
    the output to those rows; the returned arrays then have row1 - row0 rows.
    Returns (C, D) with D = sum_k |A_ik B_kj| (None if want_d is False).
    """
    lib = lib or load()
    A = np.ascontiguousarray(_as_u16(A))
    B = np.ascontiguousarray(_as_u16(B))
    M = A.shape[0] if M is None else M
    K = (A.shape[1] if A.ndim == 2 else 0) if K is None else K
    N = B.shape[1] if N is None else N
    lda = A.shape[1] if lda is None else lda
    ldb = B.shape[1] if ldb is None else ldb
    r0, r1 = (0, M) if rows is None else rows
    nr = r1 - r0
    # compute into a buffer indexed from row r0 by offsetting the pointer
    C = np.zeros((max(nr, 0), N), np.float64)
    D = np.zeros((max(nr, 0), N), np.float64) if want_d else None
    if nr <= 0 or N == 0:
        return C, D
    c_base = C.ctypes.data - r0 * N * 8
    d_base = (D.ctypes.data - r0 * N * 8) if want_d else None
    rc = lib.oracle_gemm(FMT[fmt], M, N, K, _ptr(A), lda, _ptr(B), ldb,
                         ctypes.c_void_p(c_base), ctypes.c_void_p(d_base) if want_d else None,
                         N, r0, r1)
    if rc != 0:
        raise ValueError("oracle_gemm rejected its arguments")
    return C, D


def gemm_entries(A, B, I, J, M=None, N=None, K=None, lda=None, ldb=None, fmt="bf16", lib=None):
    """Entries C_ref[I[t], J[t]] and D[I[t], J[t]], each summed in ascending k."""
    lib = lib or load()
    A = np.ascontiguousarray(_as_u16(A))
    B = np.ascontiguousarray(_as_u16(B))
    M = A.shape[0] if M is None else M
    K = A.shape[1] if K is None else K
    N = B.shape[1] if N is None else N
    lda = A.shape[1] if lda is None else lda
    ldb = B.shape[1] if ldb is None else ldb
    I = np.ascontiguousarray(I, dtype=np.int64)
    J = np.ascontiguousarray(J, dtype=np.int64)
    C = np.zeros(len(I), np.float64)
    D = np.zeros(len(I), np.float64)
    rc = lib.oracle_gemm_entries(FMT[fmt], M, N, K, _ptr(A), lda, _ptr(B), ldb,
                                 _ptr(I), _ptr(J), len(I), _ptr(C), _ptr(D))
    if rc != 0:
        raise ValueError("oracle_gemm_entries: index out of range")
    return C, D


def decode(bits, fmt="bf16", lib=None):
    """fp64 values of a uint16 array of bf16 / fp16 bit patterns."""
    lib = lib or load()
    bits = np.ascontiguousarray(_as_u16(bits))
    out = np.empty(bits.shape, np.float64)
    lib.oracle_decode(FMT[fmt], _ptr(bits), _ptr(out), bits.size)
    return out


def err_metric(C, C_ref, D):
    """max_ij |C - C_ref| / D_ij, with D_ij == 0 requiring C_ij == 0 exactly.

    C may be fp32 values or already-decoded 16-bit outputs (as fp64). NaN or
    inf in C makes the metric inf.
    """
    C = np.asarray(C, np.float64)
    C_ref = np.asarray(C_ref, np.float64)
    D = np.asarray(D, np.float64)
    if C.size == 0:
        return 0.0
    if not np.all(np.isfinite(C)):
        return float("inf")
    diff = np.abs(C - C_ref)
    zero = D == 0
    if np.any(diff[zero] != 0):
        return float("inf")
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(zero, 0.0, diff / np.where(zero, 1.0, D))
    return float(r.max())


# Acceptance bounds of the GPU path against this oracle.
TOL = {"f32": 1e-3, "bf16": 8e-3, "fp16": 1e-3}


def threads(lib=None):
    return (lib or load()).oracle_threads()
