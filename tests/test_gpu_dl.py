"""GPU parity of the direct-to-LDS tile kernels (family dl).

Every dl configuration of each shape (tile, split count, tile order) runs
through the C ABI and is checked against the fp64 oracle at the output
type's tolerance and, bit for bit, against the register-staged tile kernel
of the same tiling and split count: both multiply the same fragments in the
same k order, so any difference is a loading, swizzle or transpose-read
error. The shapes cover K tails (K not a multiple of the 64-deep k-block,
down to K = 8), ragged M and N edges, partial last stage groups and split
K, and K or N not a multiple of 8, where the plan first copies A or B into
a zero-padded form (the padding prologue). Operands that break the kernels'
alignment (an odd leading dimension, a 2-byte offset pointer) must run the
sibling tile kernel instead, and the AddMM epilogue, fp16 inputs and
column-major operands (their transposed copies) take the same path. The
decode tilings (32 or 64 rows, four waves along N) have no tile-family
counterpart: the oracle and their register-load form check them.
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
DL_SIBLING = [0, 1, 2, 3, 0, 0, 1, 2, 1, 3, 3, -1, -1, -1, -1]  # variants.h kDlCfg[i].sibling


def note(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def device():
    torch()
    ac.adaptcore_init()
    yield


def dl_candidates(M, N, K, dtype):
    return [c for c in all_candidates(M, N, K, dtype) if c["family_name"] == "dl"]


def sibling_key(key):
    """The tile-family key of a dl key: same tiling, split count, tile order
    (bit 13, the register-load form, has no tile-family counterpart); None
    for the decode tilings, which no tile kernel has."""
    cfg = (key >> 4) & 0xFF
    if DL_SIBLING[cfg] < 0:
        return None
    return (key & ~0x2FFF) | (key & (1 << 12)) | (DL_SIBLING[cfg] << 4) | ac.AC_FAMILY_TILE


SHAPES = [(300, 264, 200), (513, 640, 1000), (257, 136, 136), (1024, 1024, 1024), (96, 4096, 8192),
          (2048, 512, 64), (300, 256, 8), (130, 392, 4104), (700, 128, 520),
          # K and / or N not a multiple of 8: the padding prologue copies A / B
          (300, 263, 517), (257, 136, 133), (130, 391, 4100), (129, 255, 5), (640, 1000, 70),
          # decode-style rows (the 32 / 64-row tiles of four waves along N)
          (1, 4096, 4096), (7, 1000, 520), (33, 600, 200), (64, 264, 1000), (5, 263, 517), (16, 2048, 14336)]


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_every_dl_configuration_against_oracle_and_sibling(shape, dtype):
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=3 * M + 5 * N + K)
    ref = gemm_ref.gemm(A, B)
    cands = dl_candidates(M, N, K, dtype)
    assert cands, shape
    note("dl", shape, dtype, len(cands), "configurations")
    for c in cands:
        key = c["variant_key"]
        vals, ok = run(forced_plan(M, N, K, dtype, key), A, B, M, N, K, dtype)
        check(vals, ok, A, B, dtype, ref=ref, label="%s %s" % (shape, c))
        if sibling_key(key) is None:
            continue
        sib, ok2 = run(forced_plan(M, N, K, dtype, sibling_key(key)), A, B, M, N, K, dtype)
        assert ok2
        assert np.array_equal(vals.view(np.uint64), sib.view(np.uint64)), ("differs from the tile kernel", shape, c)


@pytest.mark.parametrize("shape", [(200, 392, 5000), (20, 1000, 9000)], ids=lambda s: "x".join(map(str, s)))
def test_integer_inputs_exact_for_every_dl_configuration(shape):
    """Integer inputs: every partial sum exact in fp32, so every split gives
    the exact integer product (the second shape: the decode tilings)."""
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=13, dist="int")
    exact = (np.rint(gemm_ref.decode(A)).astype(np.int64) @ np.rint(gemm_ref.decode(B)).astype(np.int64))
    cands = dl_candidates(M, N, K, F32)
    assert M > 64 or any(c["tile_m"] <= 64 for c in cands)
    for c in cands:
        vals, ok = run(forced_plan(M, N, K, F32, c["variant_key"]), A, B, M, N, K, F32)
        assert ok and np.array_equal(vals, exact.astype(np.float64)), c


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
@pytest.mark.parametrize("shape", [(300, 264, 520), (40, 520, 1000)], ids=lambda s: "x".join(map(str, s)))
def test_unaligned_operands_give_the_aligned_bits(shape, dtype):
    """A leading dimension that is not a multiple of 8, or an A / B pointer
    2 bytes off a 16-byte boundary, runs the configuration's register-load
    form or the register-staged tile kernel of the same tiling: the same bits
    as the direct loads on aligned operands."""
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=17)
    ref = gemm_ref.gemm(A, B)
    for c in dl_candidates(M, N, K, dtype):
        key = c["variant_key"]
        if (key >> 13) & 1:
            continue
        dl = forced_plan(M, N, K, dtype, key)
        v0, ok0 = run(dl, A, B, M, N, K, dtype)
        check(v0, ok0, A, B, dtype, ref=ref, label=str(c))
        for kw in [dict(lda=K + 3), dict(ldb=N + 4), dict(a_off=1), dict(b_off=3), dict(lda=K + 8, ldb=N + 16)]:
            v1, ok1 = run(dl, A, B, M, N, K, dtype, **kw)
            assert ok1 and np.array_equal(v1.view(np.uint64), v0.view(np.uint64)), (kw, c)


@pytest.mark.parametrize("dtype", [F16F32, F16F16], ids=["f32out", "f16out"])
def test_fp16_dl_configurations(dtype):
    M, N, K = 300, 264, 1000
    A, B = gen.operands(M, N, K, seed=19, dist="uniform_f16")
    ref = gemm_ref.gemm(A, B, fmt="fp16")
    cands = dl_candidates(M, N, K, dtype)
    assert cands
    for c in cands:
        vals, ok = run(forced_plan(M, N, K, dtype, c["variant_key"]), A, B, M, N, K, dtype)
        check(vals, ok, A, B, dtype, ref=ref, label=str(c))
        if sibling_key(c["variant_key"]) is None:
            continue
        sib, _ = run(forced_plan(M, N, K, dtype, sibling_key(c["variant_key"])), A, B, M, N, K, dtype)
        assert np.array_equal(vals.view(np.uint64), sib.view(np.uint64)), c


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
def test_addmm_through_dl_plans(dtype):
    M, N, K = 260, 392, 704
    A, B = gen.operands(M, N, K, seed=23)
    old32 = gen.uniform_f32(M, N, 24)
    old = old32 if dtype == F32 else gen.bf16_bits(old32)
    old_vals = old32.astype(np.float64) if dtype == F32 else gemm_ref.decode(old)
    bias = gen.uniform_f32(1, N, 25).reshape(-1)
    R, D = addmm_ref.addmm(A, B, old_vals, -1.25, 0.5, bias)
    for c in dl_candidates(M, N, K, dtype):
        if c["pk"] != 1:
            continue
        vals, ok = run_addmm(forced_plan(M, N, K, dtype, c["variant_key"]), A, B, M, N, K, dtype, old, -1.25, 0.5,
                             bias)
        assert ok, c
        err = gemm_ref.err_metric(vals, R, D)
        assert err <= tol(dtype), (c, err)


@pytest.mark.parametrize("layouts", [ac.AC_LAYOUT_A_COL, ac.AC_LAYOUT_B_COL, ac.AC_LAYOUT_COL_COL],
                         ids=["acol", "bcol", "colcol"])
def test_dl_column_major_operands(layouts):
    """Column-major A and / or B: the transposed copies are zero-padded
    row-major operands for the direct-to-LDS kernels; every dl configuration
    against the oracle and bit for bit against the sibling with the same
    layouts."""
    t = torch()
    M, N, K = 260, 391, 517
    a_col, b_col = bool(layouts & 1), bool(layouts & 2)
    A, B = gen.operands(M, N, K, seed=29)
    As = np.ascontiguousarray(A.T) if a_col else A
    Bs = np.ascontiguousarray(B.T) if b_col else B
    lda, ldb = (M if a_col else K), (K if b_col else N)
    R, D = layout_ref.gemm_layout(As.reshape(-1), Bs.reshape(-1), M, N, K, lda, ldb, layouts)
    cands = [c for c in all_candidates(M, N, K, F32, layouts) if c["family_name"] == "dl"]
    assert cands
    Ad = t.from_numpy(As.view(np.int16)).cuda()
    Bd = t.from_numpy(Bs.view(np.int16)).cuda()
    outs = []
    for key in [c["variant_key"] for c in cands[:16] if sibling_key(c["variant_key"]) is not None]:
        for k in (key, sibling_key(key)):
            plan = ac.adaptcore_plan_variant(M, N, K, F32, layouts, k)
            C = t.full((M, N), float("nan"), dtype=t.float32, device="cuda")
            ac.adaptcore_matmul(plan, Ad.data_ptr(), lda, Bd.data_ptr(), ldb, C.data_ptr(), N, 0)
            t.cuda.synchronize()
            outs.append(C.cpu().numpy().astype(np.float64))
        assert gemm_ref.err_metric(outs[-2], R, D) <= tol(F32), hex(key)
        assert np.array_equal(outs[-2].view(np.uint64), outs[-1].view(np.uint64)), hex(key)


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
@pytest.mark.parametrize("shape", [(300, 263, 517), (257, 136, 133), (130, 391, 4100), (640, 1000, 70), (70, 72, 9),
                                   (200, 100, 8), (129, 255, 13)], ids=lambda s: "x".join(map(str, s)))
def test_register_load_form(shape, dtype):
    """The register-load form (k_dlu: operand rows at any alignment, no
    padding prologue) of every configuration that has one, with the split
    counts and tile orders: against the oracle and bit for bit against the
    padded direct-load form of the same configuration, also with padded
    leading dimensions and 2-byte offset pointers."""
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=7 * M + N + K)
    ref = gemm_ref.gemm(A, B)
    cands = [c for c in dl_candidates(M, N, K, dtype) if (c["variant_key"] >> 13) & 1]
    assert cands, shape
    for c in cands:
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        names = ac.adaptcore_plan_kernels(plan)
        assert names[0].startswith("k_dlu<") and "k_pad16" not in names, names
        padded = forced_plan(M, N, K, dtype, c["variant_key"] & ~(1 << 13))
        for kw in [dict(), dict(lda=K + 3, ldb=N + 5, a_off=1, b_off=3)]:
            vals, ok = run(plan, A, B, M, N, K, dtype, **kw)
            check(vals, ok, A, B, dtype, ref=ref, label="%s %s %s" % (shape, kw, c))
            v2, ok2 = run(padded, A, B, M, N, K, dtype, **kw)
            assert ok2 and np.array_equal(vals.view(np.uint64), v2.view(np.uint64)), (shape, kw, c)


def test_padding_prologue_in_the_plan():
    """A dl plan of a shape with K and N not multiples of 8 lists the two
    padding copies before its kernel and reserves their workspace."""
    M, N, K = 300, 263, 517
    c = [c for c in dl_candidates(M, N, K, BF16) if not (c["variant_key"] >> 13) & 1][0]  # direct loads
    plan = forced_plan(M, N, K, BF16, c["variant_key"])
    names = ac.adaptcore_plan_kernels(plan)
    assert names[:2] == ["k_pad16", "k_pad16"] and names[2].startswith("k_dl<"), names
    d = ac.adaptcore_plan_info(plan)
    assert d["workspace_bytes"] >= 2 * (M * 520 + K * 264)
