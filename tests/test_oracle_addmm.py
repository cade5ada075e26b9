"""Pins for the AddMM oracle (CPU only).

The AddMM oracle adds a scaled input and a bias row to a scaled plain
product. These tests tie it to exact rational brute force written out here
(for C and for the acceptance scale D, with mixed-sign alpha and beta and a
bias that differs per column on non-square shapes), to the plain product it
must reduce to, and to the beta == 0 convention (C_old not read). A mutation
test checks that plausible slips in the module fail at least one pin.
"""
import importlib.util
import os
import sys
import tempfile
from fractions import Fraction

import numpy as np
import pytest

from oracle import addmm_ref
from oracle import gemm_ref
from workloads import gen

from test_oracle_gemm import exact_bf16, gamma


def _case(seed):
    rng = np.random.default_rng(300 + seed)
    M, N, K = 2 + int(rng.integers(0, 5)), 3 + int(rng.integers(0, 5)), int(rng.integers(1, 9))
    if M == N:
        N += 1  # a bias applied along the wrong axis must not fit
    A, B = gen.operands(M, N, K, seed=310 + seed)
    C_old = gen.uniform_f32(M, N, (320 + seed, 0), -2.0, 2.0).astype(np.float64)
    bias = gen.uniform_f32(1, N, (320 + seed, 1), -3.0, 3.0).reshape(-1).astype(np.float64)
    alpha = float(rng.choice([1.5, -0.75, 3.0]))
    beta = float(rng.choice([0.5, -1.25, 2.0]))
    return A, B, C_old, alpha, beta, bias


def _exact(A, B, C_old, alpha, beta, bias):
    """Exact C and D as Fractions, term by term."""
    M, K = A.shape
    N = B.shape[1]
    a = [[exact_bf16(A[i, k]) for k in range(K)] for i in range(M)]
    b = [[exact_bf16(B[k, j]) for j in range(N)] for k in range(K)]
    al, be = Fraction(alpha), Fraction(beta)
    C, D = {}, {}
    for i in range(M):
        for j in range(N):
            prod = sum((a[i][k] * b[k][j] for k in range(K)), Fraction(0))
            mag = sum((abs(a[i][k] * b[k][j]) for k in range(K)), Fraction(0))
            c = Fraction(float(C_old[i, j]))
            bj = Fraction(float(bias[j])) if bias is not None else Fraction(0)
            C[i, j] = al * prod + be * c + bj
            D[i, j] = abs(al) * mag + abs(be) * abs(c) + abs(bj)
    return C, D


def _agree(got_C, got_D, C, D, K):
    tol = Fraction(gamma(K + 3))
    for (i, j), e in C.items():
        if abs(Fraction(got_C[i, j]) - e) > tol * D[i, j]:
            return False
        if abs(Fraction(got_D[i, j]) - D[i, j]) > tol * D[i, j]:
            return False
    return True


def pin_brute_force(ar, seed=0):
    A, B, C_old, alpha, beta, bias = _case(seed)
    got_C, got_D = ar.addmm(A, B, C_old, alpha, beta, bias)
    return _agree(got_C, got_D, *_exact(A, B, C_old, alpha, beta, bias), A.shape[1])


def pin_no_bias(ar):
    A, B, C_old, alpha, beta, _ = _case(7)
    got_C, got_D = ar.addmm(A, B, C_old, alpha, beta, None)
    return _agree(got_C, got_D, *_exact(A, B, C_old, alpha, beta, None), A.shape[1])


def pin_plain_product(ar):
    """alpha = 1, beta = 0, no bias: the plain product, bit for bit."""
    A, B, C_old, _, _, _ = _case(3)
    got_C, got_D = ar.addmm(A, B, C_old, 1.0, 0.0, None)
    P, Dp = gemm_ref.gemm(A, B)
    return np.array_equal(got_C, P) and np.array_equal(got_D, Dp)


def pin_beta_zero_ignores_c_old(ar):
    """beta == 0: C_old is not read, so NaN there leaves no trace."""
    A, B, _, alpha, _, bias = _case(4)
    nan = np.full((A.shape[0], B.shape[1]), np.nan)
    got_C, got_D = ar.addmm(A, B, nan, alpha, 0.0, bias)
    if not (np.all(np.isfinite(got_C)) and np.all(np.isfinite(got_D))):
        return False
    return _agree(got_C, got_D, *_exact(A, B, np.zeros_like(nan), alpha, 0.0, bias), A.shape[1])


def pin_k_zero(ar):
    """K == 0: the product is empty and C = beta * C_old + bias exactly."""
    M, N = 3, 5
    C_old = gen.uniform_f32(M, N, (330, 0)).astype(np.float64)
    bias = gen.uniform_f32(1, N, (330, 1)).reshape(-1).astype(np.float64)
    got_C, got_D = ar.addmm(np.zeros((M, 0), np.uint16), np.zeros((0, N), np.uint16), C_old, 2.0, -0.5, bias)
    for i in range(M):
        for j in range(N):
            e = Fraction(-0.5) * Fraction(float(C_old[i, j])) + Fraction(float(bias[j]))
            d = Fraction(0.5) * abs(Fraction(float(C_old[i, j]))) + abs(Fraction(float(bias[j])))
            if Fraction(got_C[i, j]) != e or Fraction(got_D[i, j]) != d:
                return False
    return True


def pin_batched_is_per_batch(ar):
    """Every batch of the batched form equals the single form on that batch's
    matrices (padded rows, gaps between the matrices, a different C_old per
    batch, one bias), bit for bit."""
    batch, M, N, K = 3, 4, 6, 5
    lda, ldb, sa, sb = K + 2, N + 1, M * (K + 2) + 3, K * (N + 1) + 7
    A = gen.uniform_bf16(1, (batch - 1) * sa + M * lda, 350).reshape(-1)
    B = gen.uniform_bf16(1, (batch - 1) * sb + K * ldb, 351).reshape(-1)
    C_old = gen.uniform_f32(batch * M, N, 352).astype(np.float64).reshape(batch, M, N)
    bias = gen.uniform_f32(1, N, 353).reshape(-1).astype(np.float64)
    C, D = ar.batched_addmm(A, B, C_old, batch, M, N, K, lda, ldb, sa, sb, -1.5, 0.5, bias)
    for b in range(batch):
        Ab = A[b * sa:b * sa + M * lda].reshape(M, lda)[:, :K]
        Bb = B[b * sb:b * sb + K * ldb].reshape(K, ldb)[:, :N]
        Cb, Db = ar.addmm(np.ascontiguousarray(Ab), np.ascontiguousarray(Bb), C_old[b], -1.5, 0.5, bias)
        if not (np.array_equal(C[b], Cb) and np.array_equal(D[b], Db)):
            return False
    return True


def pin_grouped_is_per_group(ar):
    """Every group of the grouped form equals the single form on that group's
    rows with its own bias row (empty and truncated groups included), bit
    for bit; uncovered rows stay 0."""
    counts, rows, N, K = [3, 0, 4, -2, 9], 12, 6, 5
    stride_b, stride_bias = K * N + 3, N + 2
    A = gen.uniform_bf16(rows, K, 360)
    mats = [gen.uniform_bf16(K, N, 361 + g) for g in range(len(counts))]
    B = np.zeros(stride_b * (len(counts) - 1) + K * N, np.uint16)
    for g, m in enumerate(mats):
        B[g * stride_b:g * stride_b + K * N] = m.reshape(-1)
    C_old = gen.uniform_f32(rows, N, 366).astype(np.float64)
    bias = gen.uniform_f32(1, stride_bias * (len(counts) - 1) + N, 367).reshape(-1).astype(np.float64)
    C, D, cov = ar.grouped_addmm(A, B, counts, rows, N, K, K, N, stride_b, C_old, 0.5, -2.0, bias, stride_bias)
    bounds = [(0, 3), (3, 3), (3, 7), (7, 7), (7, 12)]  # the last group is cut at the capacity
    for g, (s, e) in enumerate(bounds):
        if e <= s:
            continue
        Cg, Dg = ar.addmm(np.ascontiguousarray(A[s:e]), mats[g], C_old[s:e], 0.5, -2.0,
                          bias[g * stride_bias:g * stride_bias + N])
        if not (np.array_equal(C[s:e], Cg) and np.array_equal(D[s:e], Dg)):
            return False
    return bool(cov.all()) and len(cov) == rows


PINS = [pin_brute_force, pin_no_bias, pin_plain_product, pin_beta_zero_ignores_c_old, pin_k_zero,
        pin_batched_is_per_batch, pin_grouped_is_per_group]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pins(pin):
    assert pin(addmm_ref)


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_tiny(seed):
    assert pin_brute_force(addmm_ref, seed)


def test_fp16_inputs():
    """fp16 bit patterns go through the fp16 decoder of the plain product."""
    A, B = gen.operands(4, 6, 5, seed=340, dist="uniform_f16")
    C_old = gen.uniform_f32(4, 6, (341, 0)).astype(np.float64)
    C, D = addmm_ref.addmm(A, B, C_old, 0.5, 1.5, None, fmt="fp16")
    P, Dp = gemm_ref.gemm(A, B, fmt="fp16")
    # scaling by powers of two and adding one term: every step exact here up to one rounding
    assert np.allclose(C, 0.5 * P + 1.5 * C_old, rtol=1e-15, atol=0)
    assert np.allclose(D, 0.5 * Dp + 1.5 * np.abs(C_old), rtol=1e-15, atol=0)


def test_entries_match_full_result():
    A, B, C_old, alpha, beta, bias = _case(11)
    C, D = addmm_ref.addmm(A, B, C_old, alpha, beta, bias)
    rng = np.random.default_rng(12)
    I = rng.integers(0, A.shape[0], 15)
    J = rng.integers(0, B.shape[1], 15)
    Ce, De = addmm_ref.addmm_entries(A, B, I, J, C_old[I, J], alpha, beta, bias[J])
    assert np.array_equal(Ce, C[I, J]) and np.array_equal(De, D[I, J])
    Ce, De = addmm_ref.addmm_entries(A, B, I, J, np.full(15, np.nan), alpha, 0.0, None)
    assert np.all(np.isfinite(Ce))


MUTATIONS = [
    ("bias dropped", "        C = C + b\n", "        C = C\n"),
    ("beta sign", "C = C + beta * Co", "C = C - beta * Co"),
    ("alpha missing from D", "D = abs(alpha) * Dp", "D = Dp"),
    ("beta term missing from D", "D = D + abs(beta) * np.abs(Co)", "D = D"),
    ("C_old read when beta is 0", "if beta != 0.0:", "if True:"),
    ("bias along the rows", "reshape(1, C.shape[1])", "reshape(C.shape[0], 1)"),
    ("alpha applied to C_old", "C = C + beta * Co", "C = C + alpha * beta * Co"),
    ("bias magnitude missing from D", "D = D + np.abs(b)", "D = D"),
    ("batched A read with the B stride", "batched_gemm(A, B, batch, M, N, K, lda, ldb, stride_a, stride_b",
     "batched_gemm(A, B, batch, M, N, K, lda, ldb, stride_b, stride_b"),
    ("batched bias along the rows", "reshape(1, 1, N)", "reshape(1, N, 1)"),
    ("grouped bias of the previous group", "b = bias[g * stride_bias:g * stride_bias + N]",
     "b = bias[max(g - 1, 0) * stride_bias:max(g - 1, 0) * stride_bias + N]"),
]


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutations_are_caught(name, old, new):
    src = open(addmm_ref.__file__).read()
    assert old in src, name
    with tempfile.TemporaryDirectory() as d:
        pkg = os.path.join(d, "oracle_mut_addmm")
        os.makedirs(pkg)
        open(os.path.join(pkg, "__init__.py"), "w").close()
        # the mutated module imports the real plain-product oracle
        with open(os.path.join(pkg, "gemm_ref.py"), "w") as f:
            f.write("from oracle.gemm_ref import *  # noqa\n")
        with open(os.path.join(pkg, "grouped_ref.py"), "w") as f:
            f.write("from oracle.grouped_ref import *  # noqa\n")
        path = os.path.join(pkg, "addmm_ref.py")
        with open(path, "w") as f:
            f.write(src.replace(old, new))
        sys.path.insert(0, d)
        try:
            import oracle_mut_addmm  # noqa: F401
            spec = importlib.util.spec_from_file_location("oracle_mut_addmm.addmm_ref", path)
            mod = importlib.util.module_from_spec(spec)
            spec.loader.exec_module(mod)
            results = []
            for pin in PINS:
                try:
                    results.append(bool(pin(mod)))
                except Exception:
                    results.append(False)
            assert not all(results), "mutation '%s' was not caught" % name
        finally:
            sys.path.remove(d)
            for m in [m for m in sys.modules if m.startswith("oracle_mut_addmm")]:
                del sys.modules[m]
