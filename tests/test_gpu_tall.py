"""GPU parity of the tall-skinny streaming kernel (family tall, N <= 32).

Every tall configuration of each shape (row block, stage count, split count)
runs through the C ABI against the fp64 oracle at the output type's
tolerance. The shapes cover N from 1 to 32 (one or two 16-column MFMA
blocks, columns past N read as zeros), ragged row blocks, K tails inside the
last 64-deep block and split K (partials summed by the reduction kernel).
Integer inputs make every partial sum exact, so every configuration must
give the exact product. B is read through its transposed copy (a prologue):
row-major B is transposed, column-major B is copied. K not a multiple of 8
takes the register-load form (k_tallu: the row-end chunk loaded as the 16
bytes ending at K and shifted down). An A whose rows are not 16-byte aligned
(odd lda, 2-byte offset pointer) at run time takes the register-load form of
the same configuration -- the same chunks in the same LDS slots, so the same
bits -- or, for configurations without one, the skinny-N kernel (checked
against the oracle). AddMM and fp16 inputs take the same kernels.
"""
import sys

import numpy as np
import pytest

import paper_2608_10803_amd as ac
from oracle import addmm_ref, gemm_ref, layout_ref
from workloads import gen

from gpu_util import all_candidates, check, forced_plan, run, run_addmm, tol, torch

pytestmark = pytest.mark.gpu

F32, BF16 = ac.AC_BF16_F32OUT, ac.AC_BF16_BF16OUT
F16F32, F16F16 = ac.AC_F16_F32OUT, ac.AC_F16_F16OUT


def note(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def device():
    torch()
    ac.adaptcore_init()
    yield


def tall_candidates(M, N, K, dtype, layouts=0):
    return [c for c in all_candidates(M, N, K, dtype, layouts) if c["family_name"] == "tall"]


SHAPES = [(1000, 10, 520), (4097, 16, 1000), (300, 1, 64), (130, 3, 8), (777, 17, 4104), (2000, 32, 1024),
          (65, 7, 200), (5000, 12, 16384), (64, 16, 72),
          # K not a multiple of 8: the register-load form
          (1000, 10, 517), (777, 17, 4100), (300, 3, 13), (5000, 12, 16279), (2000, 32, 1023), (65, 1, 9)]


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_every_tall_configuration_against_oracle(shape, dtype):
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=5 * M + 3 * N + K)
    ref = gemm_ref.gemm(A, B)
    cands = tall_candidates(M, N, K, dtype)
    assert cands, shape
    note("tall", shape, dtype, len(cands), "configurations")
    for c in cands:
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        names = ac.adaptcore_plan_kernels(plan)
        assert names[0] == "k_transpose16" and names[1].startswith("k_tallu<" if K % 8 else "k_tall<"), names
        vals, ok = run(plan, A, B, M, N, K, dtype)
        check(vals, ok, A, B, dtype, ref=ref, label="%s %s" % (shape, c))


@pytest.mark.parametrize("shape", [(3000, 14, 5000), (129, 32, 776), (3000, 14, 5003)],
                         ids=lambda s: "x".join(map(str, s)))
def test_integer_inputs_exact(shape):
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=31, dist="int")
    exact = (np.rint(gemm_ref.decode(A)).astype(np.int64) @ np.rint(gemm_ref.decode(B)).astype(np.int64))
    for c in tall_candidates(M, N, K, F32):
        vals, ok = run(forced_plan(M, N, K, F32, c["variant_key"]), A, B, M, N, K, F32)
        assert ok and np.array_equal(vals, exact.astype(np.float64)), c


def test_forms_by_k():
    """K a multiple of 8: the direct-load form; otherwise the register-load
    form (key bit 13) of the configurations that have one; K < 8: none."""
    assert all(not (c["variant_key"] >> 13) & 1 for c in tall_candidates(1000, 10, 520, BF16))
    cands = tall_candidates(1000, 10, 517, BF16)
    assert cands and all((c["variant_key"] >> 13) & 1 for c in cands)
    assert not tall_candidates(1000, 10, 4, BF16)


TALL_UNAL = [1, 1, 0, 1, 1, 0]  # variants.h kTallCfg[i].unal


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
def test_misaligned_a(dtype):
    """A with an odd leading dimension or a 2-byte offset: a configuration
    with a register-load form runs it and gives the aligned call's bits; the
    others run the skinny-N kernel and match the oracle. B's alignment does
    not matter (its transposed copy is aligned)."""
    M, N, K = 1500, 12, 2048
    A, B = gen.operands(M, N, K, seed=37)
    ref = gemm_ref.gemm(A, B)
    for c in tall_candidates(M, N, K, dtype):
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        v0, ok0 = run(plan, A, B, M, N, K, dtype)
        check(v0, ok0, A, B, dtype, ref=ref, label=str(c))
        same = TALL_UNAL[(c["variant_key"] >> 4) & 0xFF]
        for kw in [dict(lda=K + 3), dict(a_off=1), dict(ldb=N + 5, b_off=1), dict(lda=K + 8)]:
            vals, ok = run(plan, A, B, M, N, K, dtype, **kw)
            check(vals, ok, A, B, dtype, ref=ref, label="%s %s" % (kw, c))
            a_aligned = kw.get("lda", K) % 8 == 0 and kw.get("a_off", 0) == 0
            if a_aligned or same:
                assert np.array_equal(vals.view(np.uint64), v0.view(np.uint64)), (kw, c)


def test_column_major_b():
    """Column-major B (N x K in memory): its padded copy is B^T directly."""
    t = torch()
    M, N, K = 900, 11, 1000
    layouts = ac.AC_LAYOUT_B_COL
    A, B = gen.operands(M, N, K, seed=41)
    Bs = np.ascontiguousarray(B.T)
    R, D = layout_ref.gemm_layout(A.reshape(-1), Bs.reshape(-1), M, N, K, K, K, layouts)
    cands = tall_candidates(M, N, K, F32, layouts)
    assert cands
    Ad = t.from_numpy(A.view(np.int16)).cuda()
    Bd = t.from_numpy(Bs.view(np.int16)).cuda()
    for c in cands:
        plan = ac.adaptcore_plan_variant(M, N, K, F32, layouts, c["variant_key"])
        assert ac.adaptcore_plan_kernels(plan)[0] == "k_pad16"
        C = t.full((M, N), float("nan"), dtype=t.float32, device="cuda")
        ac.adaptcore_matmul(plan, Ad.data_ptr(), K, Bd.data_ptr(), K, C.data_ptr(), N, 0)
        t.cuda.synchronize()
        assert gemm_ref.err_metric(C.cpu().numpy().astype(np.float64), R, D) <= tol(F32), c


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
@pytest.mark.parametrize("K", [640, 643])
def test_addmm_through_tall_plans(dtype, K):
    M, N = 2100, 9
    A, B = gen.operands(M, N, K, seed=43)
    old32 = gen.uniform_f32(M, N, 44)
    old = old32 if dtype == F32 else gen.bf16_bits(old32)
    old_vals = old32.astype(np.float64) if dtype == F32 else gemm_ref.decode(old)
    bias = gen.uniform_f32(1, N, 45).reshape(-1)
    R, D = addmm_ref.addmm(A, B, old_vals, 0.75, -1.5, bias)
    for c in tall_candidates(M, N, K, dtype):
        vals, ok = run_addmm(forced_plan(M, N, K, dtype, c["variant_key"]), A, B, M, N, K, dtype, old, 0.75, -1.5,
                             bias)
        assert ok, c
        assert gemm_ref.err_metric(vals, R, D) <= tol(dtype), c


@pytest.mark.parametrize("dtype", [F16F32, F16F16], ids=["f32out", "f16out"])
@pytest.mark.parametrize("K", [1000, 1003])
def test_fp16_tall(dtype, K):
    M, N = 1200, 16
    A, B = gen.operands(M, N, K, seed=47, dist="uniform_f16")
    ref = gemm_ref.gemm(A, B, fmt="fp16")
    cands = tall_candidates(M, N, K, dtype)
    assert cands
    for c in cands:
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        assert ac.adaptcore_plan_kernels(plan)[1].startswith("f16::k_tall"), ac.adaptcore_plan_kernels(plan)
        vals, ok = run(plan, A, B, M, N, K, dtype)
        check(vals, ok, A, B, dtype, ref=ref, label=str(c))
