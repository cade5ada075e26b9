"""GPU parity of column-major operands (layouts AC_LAYOUT_A_COL,
AC_LAYOUT_B_COL and both) against oracle.layout_ref.

A column-major operand is copied into a row-major copy in the workspace by
the prologue kernel, then any configuration runs on the copy. Every
configuration of several ragged shapes runs for the three transposed
layouts, with padded leading dimensions (other values in the pads) and
unaligned operand pointers, and is compared element by element with the
fp64 oracle reading the same stored arrays; the default plans of larger
shapes, AddMM and the tensor binding's transposed views are covered too.
"""
import sys

import numpy as np
import pytest

import paper_2608_10803_amd as ac
from oracle import addmm_ref
from oracle import gemm_ref
from oracle import layout_ref
from workloads import gen

from gpu_util import all_candidates, check, fmt_of, forced_plan, run, run_addmm, torch

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


def stored(M, N, K, layouts, dtype, seed, pad_a=3, pad_b=5):
    """(A as stored (2-D), lda, B as stored, ldb) with other values in the pads."""
    fmt = fmt_of(dtype)
    A, B = gen.operands(M, N, K, seed=seed, dist="uniform_f16" if fmt == "fp16" else "uniform")
    mk = gen.uniform_f16 if fmt == "fp16" else gen.uniform_bf16
    if layouts & ac.AC_LAYOUT_A_COL:
        sa = mk(K, M + pad_a, (seed, 3), -9.0, 9.0)
        sa[:, :M] = A.T
        lda = M + pad_a
    else:
        sa = mk(M, K + pad_a, (seed, 3), -9.0, 9.0)
        sa[:, :K] = A
        lda = K + pad_a
    if layouts & ac.AC_LAYOUT_B_COL:
        sb = mk(N, K + pad_b, (seed, 4), -9.0, 9.0)
        sb[:, :K] = B.T
        ldb = K + pad_b
    else:
        sb = mk(K, N + pad_b, (seed, 4), -9.0, 9.0)
        sb[:, :N] = B
        ldb = N + pad_b
    return sa, lda, sb, ldb


def oracle(sa, lda, sb, ldb, M, N, K, layouts, dtype):
    return layout_ref.gemm_layout(sa, sb, M, N, K, lda, ldb, layouts, fmt=fmt_of(dtype))


LAYOUTS = [ac.AC_LAYOUT_A_COL, ac.AC_LAYOUT_B_COL, ac.AC_LAYOUT_COL_COL]
L_IDS = ["a_col", "b_col", "col_col"]
SHAPES = [(7, 5, 3), (129, 255, 257), (300, 600, 70), (3, 1000, 100), (500, 7, 300), (255, 64, 1),
          (16, 300, 1000), (64, 257, 333), (40, 6, 2000), (33, 1000, 5)]


@pytest.mark.parametrize("layouts", LAYOUTS, ids=L_IDS)
@pytest.mark.parametrize("dtype", [BF16, F16F32], ids=["bf16_bf16out", "f16_f32out"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_every_configuration(shape, dtype, layouts):
    M, N, K = shape
    sa, lda, sb, ldb = stored(M, N, K, layouts, dtype, seed=M + 2 * N + 3 * K + layouts)
    ref = oracle(sa, lda, sb, ldb, M, N, K, layouts, dtype)
    cands = all_candidates(M, N, K, dtype, layouts)
    assert cands
    note("layouts", layouts, shape, "dtype", dtype, "configurations", len(cands))
    for c in cands:
        plan = forced_plan(M, N, K, dtype, c["variant_key"], layouts)
        names = ac.adaptcore_plan_kernels(plan)
        in_place_b = c["family_name"] == "skinny_m"  # reads a column-major B directly
        if c["family_name"] == "tall":  # reads B^T: a column-major B is it already (copied padded)
            assert names[0] == ("k_pad16" if layouts & 2 else "k_transpose16"), names
        else:
            assert names.count("k_transpose16") == (layouts & 1) + (0 if in_place_b else layouts >> 1), names
        vals, ok = run(plan, sa, sb, M, N, K, dtype, lda=lda, ldb=ldb, a_off=1, b_off=1)
        check(vals, ok, None, None, dtype, ref=ref, label="%s %s" % (shape, c))


@pytest.mark.parametrize("dtype", [F32, BF16, F16F32, F16F16], ids=["bf16_f32out", "bf16_bf16out", "f16_f32out",
                                                                  "f16_f16out"])
def test_default_plans(dtype):
    """Default plans of larger shapes (persistent, split-K, skinny) for every
    transposed layout, operands without pads."""
    for (M, N, K) in [(2100, 3000, 200), (640, 1000, 4096), (4, 4096, 4096), (3000, 8, 5000)]:
        for layouts in LAYOUTS:
            sa, lda, sb, ldb = stored(M, N, K, layouts, dtype, seed=M + N + K, pad_a=0, pad_b=0)
            ref = oracle(sa, lda, sb, ldb, M, N, K, layouts, dtype)
            plan = ac.adaptcore_plan(M, N, K, dtype, layouts)
            note("layouts", layouts, (M, N, K), ac.adaptcore_plan_kernels(plan))
            vals, ok = run(plan, sa, sb, M, N, K, dtype, lda=lda, ldb=ldb)
            check(vals, ok, None, None, dtype, ref=ref, label="%s layouts %d" % ((M, N, K), layouts))


def test_copy_matches_row_major_bitwise():
    """The copy is exact: a column-major call equals the row-major call on
    the same logical operands bit for bit, on every configuration."""
    M, N, K = 129, 255, 257
    for dtype in (F32, BF16):
        A, B = gen.operands(M, N, K, seed=77)
        for layouts in LAYOUTS:
            sa = A.T.copy() if layouts & 1 else A
            sb = B.T.copy() if layouts & 2 else B
            lda = M if layouts & 1 else K
            ldb = K if layouts & 2 else N
            for c in all_candidates(M, N, K, dtype, layouts):
                key_rr = c["variant_key"] & ~(3 << 52)
                v0, ok0 = run(forced_plan(M, N, K, dtype, key_rr, 0), A, B, M, N, K, dtype)
                v1, ok1 = run(forced_plan(M, N, K, dtype, c["variant_key"], layouts), sa, sb, M, N, K, dtype,
                              lda=lda, ldb=ldb)
                assert ok0 and ok1 and np.array_equal(v0, v1), (layouts, c)


def test_addmm_and_tensor_views():
    """AddMM on column-major operands, and the tensor binding, which takes
    transposed views (contiguous columns) as column-major operands."""
    t = torch()
    M, N, K = 300, 200, 130
    for layouts in LAYOUTS:
        sa, lda, sb, ldb = stored(M, N, K, layouts, F32, seed=90 + layouts)
        c_old = gen.uniform_f32(M, N, (91, layouts))
        bias = gen.uniform_f32(1, N, (92, layouts)).reshape(-1)
        A = layout_ref.logical(sa, M, K, lda, bool(layouts & 1))
        B = layout_ref.logical(sb, K, N, ldb, bool(layouts & 2))
        ref = addmm_ref.addmm(A, B, c_old.astype(np.float64), -0.5, 2.0, bias.astype(np.float64))
        for c in all_candidates(M, N, K, F32, layouts)[:20]:
            plan = forced_plan(M, N, K, F32, c["variant_key"], layouts)
            vals, ok = run_addmm(plan, sa, sb, M, N, K, F32, c_old, -0.5, 2.0, bias, lda=lda, ldb=ldb)
            check(vals, ok, None, None, F32, ref=ref, label="addmm layouts %d %s" % (layouts, c))
    # transposed views through matmul_tensors
    A, B = gen.operands(M, N, K, seed=95)
    Ad = t.from_numpy(A.view(np.int16)).cuda().view(t.bfloat16)
    Bd = t.from_numpy(B.view(np.int16)).cuda().view(t.bfloat16)
    At = Ad.t().contiguous().t()  # same values, columns contiguous
    Bt = Bd.t().contiguous().t()
    ref = gemm_ref.gemm(A, B)
    for a, b in [(At, Bd), (Ad, Bt), (At, Bt)]:
        C = t.empty(M, N, dtype=t.float32, device="cuda")
        ac.matmul_tensors(a, b, C)
        t.cuda.synchronize()
        err = gemm_ref.err_metric(C.cpu().numpy().astype(np.float64), *ref)
        assert err <= gemm_ref.TOL["f32"], err


def test_k_zero_and_degenerate():
    """K == 0 with column-major operands writes zeros (no prologue runs);
    M == 1 and N == 1 column-major operands."""
    for layouts in LAYOUTS:
        for M, N in [(5, 7), (300, 200)]:
            plan = ac.adaptcore_plan(M, N, 0, F32, layouts)
            assert "k_transpose16" not in ac.adaptcore_plan_kernels(plan)
            vals, ok = run(plan, np.zeros((0, M), np.uint16), np.zeros((0, N), np.uint16), M, N, 0, F32,
                           lda=M if layouts & 1 else 1, ldb=1 if layouts & 2 else N)
            assert ok and np.all(vals == 0)
        for (M, N, K) in [(1, 300, 77), (300, 1, 77), (1, 1, 500)]:
            sa, lda, sb, ldb = stored(M, N, K, layouts, F32, seed=M + N + K)
            ref = oracle(sa, lda, sb, ldb, M, N, K, layouts, F32)
            vals, ok = run(ac.adaptcore_plan(M, N, K, F32, layouts), sa, sb, M, N, K, F32, lda=lda, ldb=ldb)
            check(vals, ok, None, None, F32, ref=ref, label="%s layouts %d" % ((M, N, K), layouts))
