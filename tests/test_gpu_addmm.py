"""GPU parity of AddMM: C = alpha * A * B + beta * C_old + bias through
adaptcore_addmm, against oracle.addmm_ref.

Every kernel configuration of several shapes (tile, split-K with its
reduction, stream-K with its fix-up, persistent, skinny, small-K and direct
kernels) runs on the same plans as the plain product, for all four type
combinations, and is compared element by element with the fp64 oracle under
the plain product's bars (1e-3 fp32 / fp16 output, 8e-3 bf16 output) on the
scale D = |alpha| sum|a b| + |beta| |C_old| + |bias|. Canaries around C catch
writes out of bounds; beta == 0 must not read C (NaN there stays unseen).
"""
import sys

import numpy as np
import pytest

import paper_2608_10803_amd as ac
from oracle import addmm_ref
from oracle import gemm_ref
from workloads import gen

from gpu_util import F16_SUBNORMAL_HALF_ULP, all_candidates, fmt_of, forced_plan, fp32_out, run, run_addmm, tol, \
    torch

pytestmark = pytest.mark.gpu

F32, BF16 = ac.AC_BF16_F32OUT, ac.AC_BF16_BF16OUT
F16F32, F16F16 = ac.AC_F16_F32OUT, ac.AC_F16_F16OUT
DTYPES = [F32, BF16, F16F32, F16F16]
DT_IDS = ["bf16_f32out", "bf16_bf16out", "f16_f32out", "f16_f16out"]


def note(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def device():
    torch()
    ac.adaptcore_init()
    yield


def inputs(M, N, K, dtype, seed, nan_c=False):
    """A, B bit patterns, C_old as stored (fp32 values or 16-bit patterns)
    and as numbers, and a bias row."""
    fmt = fmt_of(dtype)
    A, B = gen.operands(M, N, K, seed=seed, dist="uniform_f16" if fmt == "fp16" else "uniform")
    if fp32_out(dtype):
        stored = gen.uniform_f32(M, N, (seed, 7), -2.0, 2.0)
        if nan_c:
            stored[:] = np.nan
        vals = stored.astype(np.float64)
    else:
        mk = gen.uniform_f16 if fmt == "fp16" else gen.uniform_bf16
        stored = mk(M, N, (seed, 7), -2.0, 2.0)
        if nan_c:
            stored[:] = 0x7E00 if fmt == "fp16" else 0x7FC0
        vals = gemm_ref.decode(stored, fmt=fmt)
    bias = gen.uniform_f32(1, N, (seed, 8), -1.0, 1.0).reshape(-1)
    return A, B, stored, vals, bias


def check(vals, ok, ref, dtype, label):
    assert ok, "write outside C (canary overwritten) %s" % label
    C_ref, D = ref
    if dtype == F16F16:
        vals = np.where(np.abs(vals - C_ref) <= F16_SUBNORMAL_HALF_ULP, C_ref, vals)
    err = gemm_ref.err_metric(vals, C_ref, D)
    assert err <= tol(dtype), "err %.3g > %.3g %s" % (err, tol(dtype), label)
    return err


SHAPES = [(7, 5, 3), (129, 255, 257), (300, 600, 70), (3, 1000, 100), (500, 7, 300), (255, 64, 1)]


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_every_configuration(shape, dtype):
    M, N, K = shape
    A, B, stored, c_vals, bias = inputs(M, N, K, dtype, seed=M + 3 * N + 7 * K)
    alpha, beta = -1.5, 0.75
    ref = addmm_ref.addmm(A, B, c_vals, alpha, beta, bias, fmt=fmt_of(dtype))
    cands = all_candidates(M, N, K, dtype)
    assert cands
    note("addmm", shape, "dtype", dtype, "configurations", len(cands))
    for c in cands:
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        vals, ok = run_addmm(plan, A, B, M, N, K, dtype, stored, alpha, beta, bias)
        check(vals, ok, ref, dtype, "%s %s" % (shape, c))


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
def test_default_plans_split_and_persistent(dtype):
    """Default plans of larger shapes (split-K, skinny) and every persistent
    and stream-K configuration of one shape with more tiles than workgroups."""
    for (M, N, K) in [(2100, 3000, 200), (640, 1000, 4096), (4, 4096, 4096), (64, 64, 20000)]:
        A, B, stored, c_vals, bias = inputs(M, N, K, dtype, seed=M + N + K)
        ref = addmm_ref.addmm(A, B, c_vals, 0.5, -2.0, bias, fmt=fmt_of(dtype))
        keys = [ac.adaptcore_plan_info(ac.adaptcore_plan(M, N, K, dtype))["variant_key"]]
        if (M, N, K) == (2100, 3000, 200):
            keys += [c["variant_key"] for c in all_candidates(M, N, K, dtype)
                     if c["family_name"] in ("persist", "streamk")]
        for k in keys:
            plan = forced_plan(M, N, K, dtype, k)
            note("addmm", (M, N, K), ac.adaptcore_plan_kernels(plan))
            vals, ok = run_addmm(plan, A, B, M, N, K, dtype, stored, 0.5, -2.0, bias)
            check(vals, ok, ref, dtype, "%s %s" % ((M, N, K), hex(k)))


@pytest.mark.parametrize("dtype", DTYPES, ids=DT_IDS)
def test_beta_zero_does_not_read_c(dtype):
    """beta == 0 with NaN in C: the result is alpha * A * B + bias, finite."""
    for (M, N, K) in [(300, 600, 70), (5, 700, 3000)]:
        A, B, stored, c_vals, bias = inputs(M, N, K, dtype, seed=11 + K, nan_c=True)
        ref = addmm_ref.addmm(A, B, c_vals, 2.0, 0.0, bias, fmt=fmt_of(dtype))
        for c in all_candidates(M, N, K, dtype)[:12]:
            plan = forced_plan(M, N, K, dtype, c["variant_key"])
            vals, ok = run_addmm(plan, A, B, M, N, K, dtype, stored, 2.0, 0.0, bias)
            check(vals, ok, ref, dtype, "%s %s" % ((M, N, K), c))


def test_reduces_to_matmul_bitwise():
    """alpha = 1, beta = 0, no bias: the same bits as adaptcore_matmul on
    every configuration of one shape (the epilogue is an identity then)."""
    M, N, K = 129, 255, 257
    for dtype in DTYPES:
        A, B, stored, _, _ = inputs(M, N, K, dtype, seed=5)
        for c in all_candidates(M, N, K, dtype):
            plan = forced_plan(M, N, K, dtype, c["variant_key"])
            v1, ok1 = run(plan, A, B, M, N, K, dtype)
            v2, ok2 = run_addmm(plan, A, B, M, N, K, dtype, stored, 1.0, 0.0, None)
            assert ok1 and ok2 and np.array_equal(v1, v2), c


def test_k_zero_and_padded_operands():
    """K == 0 gives beta * C_old + bias; padded leading dimensions and
    unaligned A and B pointers leave the epilogue's indexing intact."""
    for dtype in (F32, BF16):
        for M, N in [(5, 7), (300, 200)]:
            A = np.zeros((M, 0), np.uint16)
            B = np.zeros((0, N), np.uint16)
            _, _, stored, c_vals, bias = inputs(M, N, 1, dtype, seed=M)
            ref = addmm_ref.addmm(A, B, c_vals, 3.0, -1.0, bias)
            vals, ok = run_addmm(ac.adaptcore_plan(M, N, 0, dtype), A, B, M, N, 0, dtype, stored, 3.0, -1.0, bias,
                                 lda=1)
            check(vals, ok, ref, dtype, "K=0 %s" % ((M, N),))
        M, N, K = 37, 91, 333
        A, B, _, _, bias = inputs(M, N, K, dtype, seed=9)
        ldc = N + 1
        _, _, stored, c_vals, _ = inputs(M, N, 1, dtype, seed=10)
        ref = addmm_ref.addmm(A, B, c_vals, 1.25, 0.5, bias)
        for c in all_candidates(M, N, K, dtype)[:30]:
            plan = forced_plan(M, N, K, dtype, c["variant_key"])
            vals, ok = run_addmm(plan, A, B, M, N, K, dtype, stored, 1.25, 0.5, bias, lda=K + 3, ldb=N + 5, ldc=ldc,
                                 a_off=1, b_off=3)
            check(vals, ok, ref, dtype, str(c))
