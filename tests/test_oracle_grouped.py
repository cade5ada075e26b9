"""Pins for the grouped-product oracle (CPU only).

The grouped oracle is per-group plain products over row ranges taken from
the counts. These tests tie it to things other than itself: with one shared
B the grouped product is one plain product of the covered rows; per-group
scaled identities give exact closed forms that expose any wrong group index
or row offset; empty, negative and truncated counts follow the stated
readings; permuting the groups permutes the row blocks; and tiny cases match
exact rational brute force written out here in pure Python. A mutation test
checks that plausible bookkeeping mistakes fail at least one pin.
"""
import importlib.util
import os
import tempfile
from fractions import Fraction

import numpy as np
import pytest

from oracle import gemm_ref
from oracle import grouped_ref
from workloads import gen

from test_oracle_gemm import exact_bf16, gamma


def _flat_b(mats, stride):
    """Concatenate K x N matrices at multiples of `stride` elements."""
    K, N = mats[0].shape
    out = np.zeros(stride * (len(mats) - 1) + K * N, np.uint16)
    for g, m in enumerate(mats):
        out[g * stride:g * stride + K * N] = m.reshape(-1)
    return out


def _scaled_identity_case(counts, rows, K=12, seed=21):
    """A with small integers, B_g = (g + 1) * I: exact closed form."""
    A = gen.operands(rows, K, K, seed=seed, dist="int")[0]
    mats = [gen.bf16_bits((g + 1) * np.eye(K, dtype=np.float32)) for g in range(len(counts))]
    B = _flat_b(mats, K * K + 5)
    return A, B, K * K + 5


def pin_shared_weights(gr):
    counts = [5, 0, 17, 3, 0, 0, 9]
    rows, N, K = 40, 13, 29
    A, B = gen.operands(rows, N, K, seed=31)
    C, D, cov = gr.grouped_gemm(A, B, counts, rows, N, K, K, N, 0)
    n = sum(counts)
    Cp, Dp = gemm_ref.gemm(A[:n], B)
    return np.array_equal(C[:n], Cp) and np.array_equal(D[:n], Dp) and cov[:n].all() and not cov[n:].any() \
        and not C[n:].any()


def pin_scaled_identity(gr, counts=(3, 0, 5, 1, 0, 7, 2), rows=20):
    K = 12
    A, B, sb = _scaled_identity_case(list(counts), rows, K)
    C, D, cov = gr.grouped_gemm(A, B, list(counts), rows, K, K, K, K, sb)
    a = gemm_ref.decode(A).reshape(rows, K)
    exp = np.zeros((rows, K))
    expd = np.zeros((rows, K))
    expc = np.zeros(rows, bool)
    r = 0
    for g, c in enumerate(counts):
        c = max(c, 0)
        lo, hi = min(r, rows), min(r + c, rows)
        exp[lo:hi] = (g + 1) * a[lo:hi]
        expd[lo:hi] = (g + 1) * np.abs(a[lo:hi])
        expc[lo:hi] = True
        r += c
    return np.array_equal(C, exp) and np.array_equal(D, expd) and np.array_equal(cov, expc)


def pin_negative_and_truncated(gr):
    # negative counts read as 0; rows at or past the capacity are dropped
    return (pin_scaled_identity(gr, counts=(4, -3, 5, 10), rows=12)
            and pin_scaled_identity(gr, counts=(-7, 2, 0, 3), rows=9)
            and pin_scaled_identity(gr, counts=(8, 6, 3), rows=10)
            and gr.group_rows([4, -3, 5, 10], 12) == [(0, 4), (4, 4), (4, 9), (9, 12)]
            and gr.group_rows([8, 6, 3], 10) == [(0, 8), (8, 10), (10, 10)])


def pin_permutation(gr):
    counts = [6, 2, 0, 9, 4]
    rows, N, K = 21, 10, 19
    A = gen.uniform_bf16(rows, K, 41)
    mats = [gen.uniform_bf16(K, N, 50 + g) for g in range(len(counts))]
    C, _, _ = gr.grouped_gemm(A, _flat_b(mats, K * N), counts, rows, N, K, K, N, K * N)
    perm = [3, 0, 4, 2, 1]
    starts = np.cumsum([0] + counts)
    A2 = np.concatenate([A[starts[p]:starts[p + 1]] for p in perm])
    C2, _, _ = gr.grouped_gemm(A2, _flat_b([mats[p] for p in perm], K * N), [counts[p] for p in perm], rows, N,
                               K, K, N, K * N)
    C2_back = np.concatenate([C[starts[p]:starts[p + 1]] for p in perm])
    return np.array_equal(C2, C2_back)


def brute_grouped(A, mats, counts, rows):
    """Exact rational grouped product, pure-Python loops."""
    K = A.shape[1]
    N = mats[0].shape[1]
    out = {}
    r = 0
    for g, c in enumerate(counts):
        c = max(c, 0)
        for i in range(min(r, rows), min(r + c, rows)):
            for j in range(N):
                out[(i, j)] = sum((exact_bf16(A[i, k]) * exact_bf16(mats[g][k, j]) for k in range(K)), Fraction(0))
        r += c
    return out


def pin_brute_force(gr, seed=0):
    rng = np.random.default_rng(60 + seed)
    G = int(rng.integers(1, 5))
    counts = [int(x) for x in rng.integers(0, 4, size=G)]
    rows = sum(counts) + int(rng.integers(0, 3))
    N, K = int(rng.integers(1, 6)), int(rng.integers(1, 7))
    A = gen.uniform_bf16(max(rows, 1), K, 70 + seed)[:rows]
    mats = [gen.uniform_bf16(K, N, 80 + seed * 10 + g) for g in range(G)]
    C, D, cov = gr.grouped_gemm(A, _flat_b(mats, K * N + 3), counts, rows, N, K, K, N, K * N + 3)
    E = brute_grouped(A, mats, counts, rows)
    if set(i for i, _ in E) != set(np.nonzero(cov)[0].tolist()):
        return False
    tol = Fraction(gamma(K))
    return all(abs(Fraction(C[i, j]) - e) <= tol * Fraction(D[i, j]) for (i, j), e in E.items())


def pin_batched_is_grouped_with_equal_counts(gr):
    """Contiguous batches (stride_a = M * lda) are the grouped product with
    every count equal to M."""
    batch, M, N, K = 5, 13, 11, 17
    lda, ldb = K + 2, N + 1
    A = gen.uniform_bf16(batch * M, lda, 101).reshape(-1)
    mats = [gen.uniform_bf16(K, ldb, 102 + b) for b in range(batch)]
    B = _flat_b(mats, K * ldb + 4)
    C, D = gr.batched_gemm(A, B, batch, M, N, K, lda, ldb, M * lda, K * ldb + 4)
    Cg, Dg, cov = gr.grouped_gemm(A, B, [M] * batch, batch * M, N, K, lda, ldb, K * ldb + 4)
    return cov.all() and np.array_equal(C.reshape(batch * M, N), Cg) and np.array_equal(D.reshape(batch * M, N), Dg)


def pin_batched_scaled_identity(gr):
    """B_b = (b + 1) * I with gaps between the A matrices: exact closed form."""
    batch, M, K = 4, 6, 10
    stride_a = M * K + 7
    A = np.zeros(stride_a * batch, np.uint16)
    a_vals = []
    for b in range(batch):
        Ab = gen.operands(M, K, K, seed=110 + b, dist="int")[0]
        A[b * stride_a:b * stride_a + M * K] = Ab.reshape(-1)
        a_vals.append(gemm_ref.decode(Ab))
    mats = [gen.bf16_bits((b + 1) * np.eye(K, dtype=np.float32)) for b in range(batch)]
    C, D = gr.batched_gemm(A, _flat_b(mats, K * K), batch, M, K, K, K, K, stride_a, K * K)
    return all(np.array_equal(C[b], (b + 1) * a_vals[b]) and np.array_equal(D[b], (b + 1) * np.abs(a_vals[b]))
               for b in range(batch))


def pin_batched_brute_force(gr):
    rng = np.random.default_rng(120)
    batch, M, N, K = 3, 3, 4, 5
    A = gen.uniform_bf16(batch * M, K, 121)
    mats = [gen.uniform_bf16(K, N, 122 + b) for b in range(batch)]
    C, D = gr.batched_gemm(A.reshape(-1), _flat_b(mats, K * N), batch, M, N, K, K, N, M * K, K * N)
    tol = Fraction(gamma(K))
    for b in range(batch):
        E = brute_grouped(A[b * M:(b + 1) * M], [mats[b]], [M], M)
        if not all(abs(Fraction(C[b, i, j]) - e) <= tol * Fraction(D[b, i, j]) for (i, j), e in E.items()):
            return False
    return rng is not None


PINS = [pin_shared_weights, pin_scaled_identity, pin_negative_and_truncated, pin_permutation, pin_brute_force,
        pin_batched_is_grouped_with_equal_counts, pin_batched_scaled_identity, pin_batched_brute_force]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pins(pin):
    assert pin(grouped_ref)


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_tiny(seed):
    assert pin_brute_force(grouped_ref, seed)


def test_entries_match_full_product():
    counts = [7, 0, 12, 5]
    rows, N, K = 30, 17, 23
    A = gen.uniform_bf16(rows, K + 3, 91)  # lda = K + 3
    mats = [gen.uniform_bf16(K, N + 2, 92 + g) for g in range(4)]  # ldb = N + 2
    B = _flat_b(mats, K * (N + 2) + 1)
    C, D, cov = grouped_ref.grouped_gemm(A, B, counts, rows, N, K, K + 3, N + 2, K * (N + 2) + 1)
    rng = np.random.default_rng(93)
    I = rng.integers(0, rows, 40)
    J = rng.integers(0, N, 40)
    Ce, De, ok = grouped_ref.grouped_entries(A, B, counts, rows, N, K, K + 3, N + 2, K * (N + 2) + 1, I, J)
    assert np.array_equal(ok, cov[I])
    assert np.array_equal(Ce, C[I, J]) and np.array_equal(De, D[I, J])


def test_k_zero_and_empty():
    C, D, cov = grouped_ref.grouped_gemm(np.zeros(0, np.uint16), np.zeros(0, np.uint16), [2, 3], 6, 4, 0, 1, 4, 0)
    assert not C.any() and not D.any() and cov.tolist() == [True] * 5 + [False]
    C, D, cov = grouped_ref.grouped_gemm(np.zeros(0, np.uint16), np.zeros(0, np.uint16), [], 0, 4, 3, 3, 4, 12)
    assert C.shape == (0, 4) and cov.size == 0


MUTATIONS = [
    ("no clamp of negative counts", "c = max(int(c), 0)", "c = int(c)"),
    ("start ignores the capacity", "s = min(p, rows)", "s = p"),
    ("end past the capacity", "out.append((s, min(p, rows)))", "out.append((s, p))"),
    ("off-by-one start", "Ag = A[s * lda:(e - 1) * lda + K].copy()", "Ag = A[(s + 1) * lda:e * lda + K].copy()"),
    ("wrong group matrix", "off = g * stride_b\n", "off = max(g - 1, 0) * stride_b\n"),
    ("batch ignores stride_a", "a0 = b * stride_a\n", "a0 = b * M * lda\n"),
]


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutations_are_caught(name, old, new):
    src = open(grouped_ref.__file__).read()
    assert old in src, name
    with tempfile.TemporaryDirectory() as d:
        pkg = os.path.join(d, "oracle_mut")
        os.makedirs(pkg)
        # the mutated module imports the real plain-product oracle
        open(os.path.join(pkg, "__init__.py"), "w").close()
        with open(os.path.join(pkg, "gemm_ref.py"), "w") as f:
            f.write("from oracle.gemm_ref import *  # noqa\n")
        path = os.path.join(pkg, "grouped_ref.py")
        with open(path, "w") as f:
            f.write(src.replace(old, new))
        import sys
        sys.path.insert(0, d)
        try:
            spec = importlib.util.spec_from_file_location("oracle_mut.grouped_ref", path,
                                                          submodule_search_locations=None)
            import oracle_mut  # noqa: F401
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
            for m in [m for m in sys.modules if m.startswith("oracle_mut")]:
                del sys.modules[m]
