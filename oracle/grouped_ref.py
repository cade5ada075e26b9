"""Grouped product (GroupMM) oracle -- TEST INFRASTRUCTURE ONLY.

Only tests, the smoke check and the benchmark's CPU-baseline leg may import
this module; it shares no code with the GPU library.

The paper runs its end-to-end workloads with the dense products of the model
(MatMul, AddMM, GroupMM, BatchMM) replaced by its own (Section 6.5, and the
operator scope stated in Section 7); MoE routing is the paper's example of
GEMM dimensions that change at run time (Section 2.2). A grouped product
runs one dense product per group, all groups sharing N and K. It is read here
in the contiguous form an MoE layer produces after sorting tokens by expert:

  * A holds the rows of all groups one after another (row-major, lda); group
    g owns `counts[g]` consecutive rows, starting after the rows of groups
    0 .. g-1;
  * group g multiplies its rows by its own K x N matrix B_g, which starts
    `stride_b` elements after B_{g-1} (row-major, ldb; stride_b = 0 shares
    one B between all groups);
  * C has the same row order as A (ldc): C[rows of g] = A[rows of g] * B_g.

Device-resident counts cannot be validated by the host, so two readings make
every count array well defined: a negative count is read as 0, and rows at
or past the capacity `rows` (the rows A and C were allocated with) are
dropped -- group g covers rows [min(P_{g-1}, rows), min(P_g, rows)) with P_g
the running sum of the non-negative counts. Rows not covered by any group
are not part of the result (the GPU leaves them untouched).

A batched product (BatchMM, named beside GroupMM in the same sections) is
read as the strided form: batch b multiplies the M x K matrix at
A + b * stride_a (lda) by the K x N matrix at B + b * stride_b (ldb) into the
M x N matrix at C + b * stride_c (ldc); batched_gemm writes it out.

Parity pins: tests/test_oracle_grouped.py (shared weights reduce to one plain
product, per-group scaled identities in exact arithmetic, empty, negative and
truncated counts, group permutation, pure-Python brute force on tiny inputs;
for the batched form: contiguous batches equal the grouped product with equal
counts, per-batch scaled identities, brute force).
"""
import numpy as np

from . import gemm_ref


def group_rows(counts, rows):
    """[(start, end)] row range of every group under the readings above."""
    out = []
    p = 0
    for c in counts:
        c = max(int(c), 0)
        s = min(p, rows)
        p += c
        out.append((s, min(p, rows)))
    return out


def group_b(B, g, K, N, ldb, stride_b):
    """The K x N matrix of group g inside the flat uint16 array B."""
    off = g * stride_b
    if K == 0 or N == 0:
        return np.zeros((K, N), np.uint16)
    if off + (K - 1) * ldb + N > B.size:
        raise ValueError("B does not hold group %d" % g)
    return np.lib.stride_tricks.as_strided(B[off:], shape=(K, N), strides=(ldb * 2, 2))


def grouped_gemm(A, B, counts, rows, N, K, lda, ldb, stride_b, fmt="bf16", lib=None):
    """C_ref, D and the covered-row mask of the grouped product.

    A: uint16 array of at least rows * lda elements (flattened row-major);
    B: flat uint16 array holding every group's matrix at multiples of
    stride_b. Returns (C, D, covered) with C, D of shape (rows, N) in fp64
    (uncovered rows are 0 in both) and covered a bool array of length rows.
    """
    A = np.ascontiguousarray(A).reshape(-1)
    B = np.ascontiguousarray(B).reshape(-1)
    C = np.zeros((rows, N), np.float64)
    D = np.zeros((rows, N), np.float64)
    covered = np.zeros(rows, bool)
    for g, (s, e) in enumerate(group_rows(counts, rows)):
        if e <= s:
            continue
        covered[s:e] = True
        if K == 0 or N == 0:
            continue
        Ag = A[s * lda:(e - 1) * lda + K].copy()
        Ag = np.concatenate([Ag, np.zeros(lda - K, np.uint16)]).reshape(e - s, lda)
        Bg = np.ascontiguousarray(group_b(B, g, K, N, ldb, stride_b))
        Cg, Dg = gemm_ref.gemm(Ag, Bg, M=e - s, N=N, K=K, lda=lda, ldb=N, fmt=fmt, lib=lib)
        C[s:e] = Cg
        D[s:e] = Dg
    return C, D, covered


def grouped_entries(A, B, counts, rows, N, K, lda, ldb, stride_b, I, J, fmt="bf16", lib=None):
    """Entries (I[t], J[t]) of the grouped product, each computed on its own
    from its group's A row and B column. Entries of uncovered rows are
    reported through the returned mask (False) with value 0."""
    bounds = group_rows(counts, rows)
    starts = np.array([s for s, _ in bounds], np.int64)
    ends = np.array([e for _, e in bounds], np.int64)
    C = np.zeros(len(I), np.float64)
    D = np.zeros(len(I), np.float64)
    ok = np.zeros(len(I), bool)
    A = np.ascontiguousarray(A).reshape(-1)
    B = np.ascontiguousarray(B).reshape(-1)
    for t, (i, j) in enumerate(zip(I, J)):
        hit = np.nonzero((starts <= i) & (i < ends))[0]
        if len(hit) == 0:
            continue
        g = int(hit[0])
        ok[t] = True
        if K == 0:
            continue
        Ar = A[i * lda:i * lda + K].reshape(1, K)
        off = g * stride_b + int(j)
        if off + (K - 1) * ldb >= B.size:
            raise ValueError("B does not hold group %d" % g)
        Bc = np.ascontiguousarray(B[off:off + (K - 1) * ldb + 1:ldb]).reshape(K, 1)
        c, d = gemm_ref.gemm_entries(Ar, Bc, [0], [0], M=1, N=1, K=K, lda=K, ldb=1, fmt=fmt, lib=lib)
        C[t], D[t] = c[0], d[0]
    return C, D, ok


def batched_gemm(A, B, batch, M, N, K, lda, ldb, stride_a, stride_b, fmt="bf16", lib=None):
    """C_ref and D of a strided batched product, shape (batch, M, N) in fp64.
    A and B are flat uint16 arrays holding every batch's matrix."""
    A = np.ascontiguousarray(A).reshape(-1)
    B = np.ascontiguousarray(B).reshape(-1)
    C = np.zeros((batch, M, N), np.float64)
    D = np.zeros((batch, M, N), np.float64)
    if M == 0 or N == 0 or K == 0:
        return C, D
    for b in range(batch):
        a0 = b * stride_a
        if a0 + (M - 1) * lda + K > A.size:
            raise ValueError("A does not hold batch %d" % b)
        Ab = np.lib.stride_tricks.as_strided(A[a0:], shape=(M, K), strides=(lda * 2, 2))
        Bb = np.ascontiguousarray(group_b(B, b, K, N, ldb, stride_b))
        C[b], D[b] = gemm_ref.gemm(np.ascontiguousarray(Ab), Bb, fmt=fmt, lib=lib)
    return C, D
