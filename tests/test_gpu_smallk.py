"""GPU parity of the small-K kernels (K <= 16, family smallk).

Rows of fewer than 1024 columns run k_smallk (a thread: 8 columns of a run
of rows). Wider rows run k_smallk_win: a workgroup owns a band of rows and
1984 columns, computes 64 more columns to their left, and per row stores
the window that starts at the 128-byte line boundary at or before its first
column, shifted there through LDS. Both form every sum in the same order,
so integer inputs give the exact product and real inputs match the fp64
oracle at the output type's tolerance. The shapes cover one and several
windows per row, a last window that ends inside a line, bands that end
before R rows, K below the kernel's bound, and -- through the leading
dimension of C -- rows whose starts fall at every offset within a line.
The canaries around C catch any write outside the rows' N columns. AddMM
takes the same kernels (its epilogue at store time in the window kernel).
"""
import sys

import numpy as np
import pytest

import paper_2608_10803_amd as ac
from oracle import addmm_ref, gemm_ref
from workloads import gen

from gpu_util import all_candidates, check, forced_plan, run, run_addmm, tol, torch

pytestmark = pytest.mark.gpu

F32, BF16 = ac.AC_BF16_F32OUT, ac.AC_BF16_BF16OUT
WIN_MIN_N = 1024  # narrower rows take k_smallk


def note(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def device():
    torch()
    ac.adaptcore_init()
    yield


SHAPES = [(5000, 8, 4), (3000, 16, 13), (4099, 300, 1), (2500, 100, 7), (7, 5, 3), (777, 1000, 8),
          (777, 3000, 8), (1001, 2049, 16), (64, 4100, 9), (33, 1024, 2), (1, 5000, 5), (130, 3969, 3),
          (257, 1984, 12)]


def smallk_candidates(M, N, K, dtype):
    return [c for c in all_candidates(M, N, K, dtype) if c["family_name"] == "smallk"]


def test_kernel_by_width():
    for M, N, K in SHAPES:
        for c in smallk_candidates(M, N, K, BF16):
            names = ac.adaptcore_plan_kernels(forced_plan(M, N, K, BF16, c["variant_key"]))
            want = "k_smallk_win<" if N >= WIN_MIN_N else "k_smallk<"
            assert len(names) == 1 and names[0].startswith(want), (M, N, K, names)


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_smallk_against_oracle(shape, dtype):
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=3 * M + N + 7 * K)
    ref = gemm_ref.gemm(A, B)
    cands = smallk_candidates(M, N, K, dtype)
    assert cands, shape
    for c in cands:
        note("smallk", shape, dtype, c["tile_m"], ac.adaptcore_plan_kernels(forced_plan(M, N, K, dtype,
                                                                                         c["variant_key"])))
        vals, ok = run(forced_plan(M, N, K, dtype, c["variant_key"]), A, B, M, N, K, dtype)
        check(vals, ok, A, B, dtype, ref=ref, label="%s %s" % (shape, c))


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_smallk_integer_inputs_exact(shape):
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=59, dist="int")
    exact = (np.rint(gemm_ref.decode(A)).astype(np.int64) @ np.rint(gemm_ref.decode(B)).astype(np.int64))
    for c in smallk_candidates(M, N, K, F32):
        vals, ok = run(forced_plan(M, N, K, F32, c["variant_key"]), A, B, M, N, K, F32)
        assert ok and np.array_equal(vals, exact.astype(np.float64)), c


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
@pytest.mark.parametrize("N", [1000, 2500])
def test_smallk_strides_and_offsets(N, dtype):
    """Odd leading dimensions and 2-byte offsets of A and B, and leading
    dimensions of C that move each row's start within a line: every call
    gives the bits of the packed call."""
    M, K = 700, 5
    A, B = gen.operands(M, N, K, seed=61)
    ref = gemm_ref.gemm(A, B)
    for c in smallk_candidates(M, N, K, dtype):
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        v0, ok0 = run(plan, A, B, M, N, K, dtype)
        check(v0, ok0, A, B, dtype, ref=ref, label=str(c))
        for kw in [dict(lda=K + 3), dict(a_off=1), dict(ldb=N + 5, b_off=1), dict(ldc=N + 1), dict(ldc=N + 37),
                   dict(ldc=N + 64)]:
            vals, ok = run(plan, A, B, M, N, K, dtype, **kw)
            assert ok and np.array_equal(vals.view(np.uint64), v0.view(np.uint64)), (kw, c)


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
@pytest.mark.parametrize("N", [700, 2100])
def test_smallk_addmm(N, dtype):
    M, K = 1500, 6
    A, B = gen.operands(M, N, K, seed=67)
    old32 = gen.uniform_f32(M, N, 68)
    old = old32 if dtype == F32 else gen.bf16_bits(old32)
    old_vals = old32.astype(np.float64) if dtype == F32 else gemm_ref.decode(old)
    bias = gen.uniform_f32(1, N, 69).reshape(-1)
    R, D = addmm_ref.addmm(A, B, old_vals, 0.5, 2.0, bias)
    for c in smallk_candidates(M, N, K, dtype):
        vals, ok = run_addmm(forced_plan(M, N, K, dtype, c["variant_key"]), A, B, M, N, K, dtype, old, 0.5, 2.0,
                             bias)
        assert ok, c
        assert gemm_ref.err_metric(vals, R, D) <= tol(dtype), c


@pytest.mark.parametrize("dtype", [ac.AC_F16_F32OUT, ac.AC_F16_F16OUT], ids=["f32out", "f16out"])
@pytest.mark.parametrize("shape", [(900, 700, 7), (700, 2500, 13), (300, 4100, 16)],
                         ids=lambda s: "x".join(map(str, s)))
def test_smallk_fp16_inputs(shape, dtype):
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=71, dist="uniform_f16")
    ref = gemm_ref.gemm(A, B, fmt="fp16")
    cands = smallk_candidates(M, N, K, dtype)
    assert cands
    for c in cands:
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        assert ac.adaptcore_plan_kernels(plan)[0].startswith("f16::k_smallk"), ac.adaptcore_plan_kernels(plan)
        vals, ok = run(plan, A, B, M, N, K, dtype)
        check(vals, ok, A, B, dtype, ref=ref, label=str(c))
