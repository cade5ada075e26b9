"""Pins for the GEMM oracle (CPU only).

The oracle is the plain definition C = A * B in fp64. These tests tie it to
things other than itself: exact rational brute force, an independent BLAS
product within the classical error bound, exact integer arithmetic, and the
identities of the product (identity matrix, all-ones, transposition, outer
products, permutations). A mutation test checks that plausible mistakes in
the oracle's C source are caught by these pins.
"""
import os
import shutil
import subprocess
import tempfile
from fractions import Fraction

import numpy as np
import pytest

from oracle import gemm_ref
from oracle import build as obuild
from workloads import gen

U = 2.0 ** -53


def gamma(k):
    return k * U / (1 - k * U)


def exact_bf16(bits):
    """Exact rational value of bf16 bits, independent of the oracle's decoder."""
    b = int(bits)
    sign = -1 if b & 0x8000 else 1
    e = (b >> 7) & 0xFF
    f = b & 0x7F
    if e == 0:
        return sign * Fraction(f, 2 ** 133)  # f * 2^-7 * 2^-126
    assert e != 0xFF
    return sign * Fraction(f + 128, 128) * Fraction(2) ** (e - 127)


def brute_force(A, B):
    M, K = A.shape
    N = B.shape[1]
    a = [[exact_bf16(A[i, k]) for k in range(K)] for i in range(M)]
    b = [[exact_bf16(B[k, j]) for j in range(N)] for k in range(K)]
    return [[sum((a[i][k] * b[k][j] for k in range(K)), Fraction(0)) for j in range(N)]
            for i in range(M)]


@pytest.mark.parametrize("seed", range(6))
def test_p1_brute_force_tiny(seed):
    rng = np.random.default_rng(100 + seed)
    M, N, K = (int(x) for x in rng.integers(1, 9, size=3))
    A, B = gen.operands(M, N, K, seed=200 + seed)
    C, D = gemm_ref.gemm(A, B)
    E = brute_force(A, B)
    g = gamma(K)
    for i in range(M):
        for j in range(N):
            assert abs(Fraction(C[i, j]) - E[i][j]) <= Fraction(g) * Fraction(D[i, j])
            absum = sum(abs(exact_bf16(A[i, k]) * exact_bf16(B[k, j])) for k in range(K))
            assert abs(Fraction(D[i, j]) - absum) <= Fraction(g) * absum


def test_p1b_blas_moderate():
    M, N, K = 67, 45, 301
    A, B = gen.operands(M, N, K, seed=7)
    C, D = gemm_ref.gemm(A, B)
    a = A.astype(np.uint32) << 16
    b = B.astype(np.uint32) << 16
    Af = a.view(np.float32).astype(np.float64)
    Bf = b.view(np.float32).astype(np.float64)
    R = Af @ Bf
    Dn = np.abs(Af) @ np.abs(Bf)
    assert np.all(np.abs(C - R) <= 2 * gamma(K) * Dn)
    assert np.allclose(D, Dn, rtol=4 * gamma(K), atol=0)


def test_p2_identity():
    M, K = 37, 29
    A = gen.uniform_bf16(M, K, 11)
    I = gen.bf16_bits(np.eye(K, dtype=np.float32))
    C, _ = gemm_ref.gemm(A, I)
    assert np.array_equal(C, gemm_ref.decode(A))


@pytest.mark.parametrize("K", [1, 7, 64, 1000])
def test_p3_all_ones(K):
    A = gen.bf16_bits(np.ones((5, K), np.float32))
    B = gen.bf16_bits(np.ones((K, 9), np.float32))
    C, D = gemm_ref.gemm(A, B)
    assert np.all(C == K) and np.all(D == K)


def test_p4_transposition():
    M, N, K = 23, 31, 47
    A, B = gen.operands(M, N, K, seed=12)
    C1, _ = gemm_ref.gemm(A, B)
    C2, _ = gemm_ref.gemm(np.ascontiguousarray(B.T), np.ascontiguousarray(A.T))
    assert np.array_equal(C1, C2.T)


def test_p5_integer_exact():
    M, N, K = 40, 33, 517
    A, B = gen.operands(M, N, K, seed=13, dist="int")
    C, _ = gemm_ref.gemm(A, B)
    Ai = np.rint(gemm_ref.decode(A)).astype(np.int64)
    Bi = np.rint(gemm_ref.decode(B)).astype(np.int64)
    assert np.array_equal(C, (Ai @ Bi).astype(np.float64))


def test_p6_outer_product_and_permutation():
    a = gen.uniform_bf16(19, 1, 14)
    b = gen.uniform_bf16(1, 23, 15)
    C, _ = gemm_ref.gemm(a, b)
    assert np.array_equal(C, np.outer(gemm_ref.decode(a)[:, 0], gemm_ref.decode(b)[0]))
    perm = np.random.default_rng(16).permutation(30)
    P = np.zeros((30, 30), np.float32)
    P[np.arange(30), perm] = 1.0
    B = gen.uniform_bf16(30, 17, 17)
    C, _ = gemm_ref.gemm(gen.bf16_bits(P), B)
    assert np.array_equal(C, gemm_ref.decode(B)[perm])


def test_rows_entries_and_strides_agree():
    M, N, K = 21, 18, 33
    A, B = gen.operands(M, N, K, seed=18)
    C, D = gemm_ref.gemm(A, B)
    Cr, Dr = gemm_ref.gemm(A, B, rows=(5, 12))
    assert np.array_equal(Cr, C[5:12]) and np.array_equal(Dr, D[5:12])
    I = np.array([0, 20, 7, 3]); J = np.array([17, 0, 9, 3])
    Ce, De = gemm_ref.gemm_entries(A, B, I, J)
    assert np.array_equal(Ce, C[I, J]) and np.array_equal(De, D[I, J])
    # padded leading dimensions select the same sub-matrices
    Ap = np.zeros((M, K + 5), np.uint16); Ap[:, :K] = A
    Bp = np.zeros((K, N + 3), np.uint16); Bp[:, :N] = B
    Cp, _ = gemm_ref.gemm(Ap, Bp, M=M, N=N, K=K, lda=K + 5, ldb=N + 3)
    assert np.array_equal(Cp, C)


def test_k_zero_and_empty():
    A = np.zeros((3, 0), np.uint16)
    B = np.zeros((0, 4), np.uint16)
    C, D = gemm_ref.gemm(A, B, K=0)
    assert C.shape == (3, 4) and np.all(C == 0) and np.all(D == 0)
    C, _ = gemm_ref.gemm(np.zeros((0, 5), np.uint16), gen.uniform_bf16(5, 4, 1))
    assert C.shape == (0, 4)


def test_decode_exhaustive():
    bits = np.arange(65536, dtype=np.uint16)
    got = gemm_ref.decode(bits, "bf16")
    ref = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    assert np.array_equal(got[~np.isnan(ref)], ref[~np.isnan(ref)])
    got = gemm_ref.decode(bits, "fp16")
    ref = bits.view(np.float16).astype(np.float64)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    assert np.array_equal(got[~np.isnan(ref)], ref[~np.isnan(ref)])


def test_err_metric():
    C_ref = np.array([[1.0, 2.0], [0.0, -1.0]])
    D = np.array([[2.0, 4.0], [0.0, 1.0]])
    assert gemm_ref.err_metric(C_ref, C_ref, D) == 0.0
    assert gemm_ref.err_metric(C_ref + [[0.002, 0], [0, 0]], C_ref, D) == pytest.approx(0.001)
    assert gemm_ref.err_metric(C_ref + [[0, 0], [1e-30, 0]], C_ref, D) == float("inf")
    assert gemm_ref.err_metric(C_ref * np.nan, C_ref, D) == float("inf")


def test_generators_deterministic_and_rne():
    a1 = gen.uniform_bf16(8, 8, 3)
    a2 = gen.uniform_bf16(8, 8, 3)
    assert np.array_equal(a1, a2)
    # bf16 rounding: exactly representable values are unchanged, ties go to even
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -7], np.float32)
    got = gemm_ref.decode(gen.bf16_bits(x))
    assert list(got) == [1.0, 1.0, 1.0 + 2 ** -6, -2.5, 1.0 + 2 ** -7]


def test_sweep_reading():
    shapes, rej = gen.sweep(return_rejections=True)
    assert len(shapes) == 2000 and rej == 173
    assert all(1 <= d <= 100000 for s in shapes for d in s)
    assert all(gen.sweep_accepts(*s) for s in shapes)
    assert shapes == gen.sweep()


def test_moe_counts():
    cs = gen.moe_counts(steps=10)
    assert all(int(c.sum()) == 8192 and len(c) == 64 for c in cs)
    small = np.mean([np.mean(c <= 10) for c in cs])
    assert small > 0.5  # many experts with 0-10 tokens


# ---- mutation test: plausible mistakes in the oracle must fail a pin --------

MUTATIONS = [
    ("drop last k", "for (int64_t k = 0; k < K; ++k) {\n            double a",
     "for (int64_t k = 0; k < K - 1; ++k) {\n            double a"),
    ("transposed B index", "const uint16_t *brow = B + (size_t)k * (size_t)ldb;",
     "const uint16_t *brow = B + (size_t)k;"),
    ("sign flip", "c[j] += p;", "c[j] -= p;"),
    ("bf16 decode shift", "((uint32_t)h) << 16", "((uint32_t)h) << 15"),
    ("abs-sum without fabs", "if (d) d[j] += fabs(p);", "if (d) d[j] += p;"),
]


def _pins(lib):
    """A compact run of the pins above against a given oracle library."""
    fails = []
    A, B = gen.operands(5, 6, 7, seed=200)
    C, D = gemm_ref.gemm(A, B, lib=lib)
    E = brute_force(A, B)
    if any(abs(Fraction(C[i, j]) - E[i][j]) > Fraction(gamma(7)) * Fraction(abs(D[i, j]) + 1e-300)
           for i in range(5) for j in range(6)):
        fails.append("brute")
    Ai, Bi = gen.operands(9, 8, 11, seed=13, dist="int")
    Ci, _ = gemm_ref.gemm(Ai, Bi, lib=lib)
    ia = np.rint(gemm_ref.decode(Ai)).astype(np.int64)
    ib = np.rint(gemm_ref.decode(Bi)).astype(np.int64)
    if not np.array_equal(Ci, (ia @ ib).astype(np.float64)):
        fails.append("int")
    if not np.all(D >= np.abs(C) - 1e-12):
        fails.append("abs")
    return fails


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("name,old,new", MUTATIONS)
def test_mutations_are_caught(name, old, new):
    src = open(obuild.SRC).read()
    assert old in src, name
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, "gemm_ref.c")
        with open(path, "w") as f:
            f.write(src.replace(old, new))
        out = os.path.join(d, "libmut.so")
        subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-shared", "-fPIC", path, "-o", out, "-lm"],
                       check=True, capture_output=True)
        lib = gemm_ref.load(out)
        assert _pins(lib), "mutation '%s' was not caught" % name
    assert not _pins(gemm_ref.load())
