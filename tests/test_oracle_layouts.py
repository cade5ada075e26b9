"""Pins for the operand-layout oracle (CPU only).

The layout oracle reads the logical A and B out of their stored arrays and
calls the plain-product oracle. These tests tie the index rules to exact
rational brute force that indexes the stored arrays itself (A column-major:
element (i, k) at i + k * lda; B column-major: element (k, j) at
k + j * ldb), for all four layouts with padded leading dimensions on
non-square shapes, and to the transposition identity (a column-major operand
stored as the row-major transpose gives the row-major product bit for bit).
A mutation test checks that slips in the index rules fail a pin.
"""
import importlib.util
import os
import sys
import tempfile
from fractions import Fraction

import numpy as np
import pytest

from oracle import gemm_ref
from oracle import layout_ref
from workloads import gen

from test_oracle_gemm import exact_bf16, gamma


def _stored(seed, M, N, K, layouts, pad_a=3, pad_b=2):
    """Stored arrays (flat, padded, garbage in the pads) and leading dims."""
    A, B = gen.operands(M, N, K, seed=seed)
    if layouts & 1:
        lda = M + pad_a
        mem_a = gen.uniform_bf16(K, lda, (seed, 3), -9.0, 9.0)  # pads hold other values
        mem_a[:, :M] = A.T
    else:
        lda = K + pad_a
        mem_a = gen.uniform_bf16(M, lda, (seed, 3), -9.0, 9.0)
        mem_a[:, :K] = A
    if layouts & 2:
        ldb = K + pad_b
        mem_b = gen.uniform_bf16(N, ldb, (seed, 4), -9.0, 9.0)
        mem_b[:, :K] = B.T
    else:
        ldb = N + pad_b
        mem_b = gen.uniform_bf16(K, ldb, (seed, 4), -9.0, 9.0)
        mem_b[:, :N] = B
    return mem_a.reshape(-1), mem_b.reshape(-1), lda, ldb


def _brute(mem_a, mem_b, M, N, K, lda, ldb, layouts):
    def a(i, k):
        return exact_bf16(mem_a[i + k * lda] if layouts & 1 else mem_a[i * lda + k])

    def b(k, j):
        return exact_bf16(mem_b[k + j * ldb] if layouts & 2 else mem_b[k * ldb + j])

    return {(i, j): sum((a(i, k) * b(k, j) for k in range(K)), Fraction(0)) for i in range(M) for j in range(N)}


def pin_brute_force(lr, seed=0):
    rng = np.random.default_rng(400 + seed)
    for layouts in range(4):
        M, N, K = 2 + int(rng.integers(0, 5)), 2 + int(rng.integers(0, 5)), 1 + int(rng.integers(0, 7))
        if len({M, N, K}) < 3:
            M, N, K = 3, 5, 4
        mem_a, mem_b, lda, ldb = _stored(410 + seed, M, N, K, layouts)
        C, D = lr.gemm_layout(mem_a, mem_b, M, N, K, lda, ldb, layouts)
        E = _brute(mem_a, mem_b, M, N, K, lda, ldb, layouts)
        tol = Fraction(gamma(K))
        for (i, j), e in E.items():
            if abs(Fraction(C[i, j]) - e) > tol * Fraction(D[i, j]):
                return False
    return True


def pin_transposed_storage(lr):
    """Storing A^T (and B^T) row-major and reading it column-major gives the
    plain row-major product, bit for bit."""
    M, N, K = 13, 7, 29
    A, B = gen.operands(M, N, K, seed=420)
    C0, D0 = gemm_ref.gemm(A, B)
    for layouts in range(4):
        mem_a = np.ascontiguousarray(A.T if layouts & 1 else A).reshape(-1)
        mem_b = np.ascontiguousarray(B.T if layouts & 2 else B).reshape(-1)
        lda = M if layouts & 1 else K
        ldb = K if layouts & 2 else N
        C, D = lr.gemm_layout(mem_a, mem_b, M, N, K, lda, ldb, layouts)
        if not (np.array_equal(C, C0) and np.array_equal(D, D0)):
            return False
    return True


PINS = [pin_brute_force, pin_transposed_storage]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pins(pin):
    assert pin(layout_ref)


@pytest.mark.parametrize("seed", range(4))
def test_brute_force_tiny(seed):
    assert pin_brute_force(layout_ref, seed)


def test_short_array_is_rejected():
    with pytest.raises(ValueError):
        layout_ref.logical(np.zeros(10, np.uint16), 3, 4, 3, True)  # needs 2 + 3 * 3 + 1 = 12 elements
    assert layout_ref.logical(np.arange(12, dtype=np.uint16), 3, 4, 3, True)[2, 3] == 11


MUTATIONS = [
    ("column-major strides swapped", "last, strides = (rows - 1) + (cols - 1) * ld, (2, 2 * ld)",
     "last, strides = (rows - 1) + (cols - 1) * ld, (2 * ld, 2)"),
    ("row-major reads the transpose", "last, strides = (rows - 1) * ld + (cols - 1), (2 * ld, 2)",
     "last, strides = (rows - 1) * ld + (cols - 1), (2, 2 * ld)"),
    ("B tested with the A bit", "bool(layouts & B_COL)", "bool(layouts & A_COL)"),
    ("A tested with the B bit", "bool(layouts & A_COL))", "bool(layouts & B_COL))"),
    ("B read with lda", "B = logical(B_mem, K, N, ldb,", "B = logical(B_mem, K, N, lda,"),
]


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutations_are_caught(name, old, new):
    src = open(layout_ref.__file__).read()
    assert old in src, name
    with tempfile.TemporaryDirectory() as d:
        pkg = os.path.join(d, "oracle_mut_layout")
        os.makedirs(pkg)
        open(os.path.join(pkg, "__init__.py"), "w").close()
        with open(os.path.join(pkg, "gemm_ref.py"), "w") as f:
            f.write("from oracle.gemm_ref import *  # noqa\n")
        path = os.path.join(pkg, "layout_ref.py")
        with open(path, "w") as f:
            f.write(src.replace(old, new))
        sys.path.insert(0, d)
        try:
            import oracle_mut_layout  # noqa: F401
            spec = importlib.util.spec_from_file_location("oracle_mut_layout.layout_ref", path)
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
            for m in [m for m in sys.modules if m.startswith("oracle_mut_layout")]:
                del sys.modules[m]
