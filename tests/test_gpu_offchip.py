"""GPU parity of the off-chip accumulation kernel (family offchip: the
SingleCoreSplitK and HybridSplitK templates).

A workgroup owns a super-tile of two vertically adjacent 256 x 256 tiles,
takes its k1-slices of K in order, and flushes both tiles' partial sums to
the workspace after every slice; the reduction kernel adds the slices. Every
tile of every slice is computed exactly as the direct-to-LDS tile kernel's
split-K plan with the same slices computes it, so each configuration must
give that plan's bits, and match the fp64 oracle at the output type's
tolerance. The shapes cover an odd number of tile rows (a super-tile with
one tile), ragged edges, K tails inside the last slice, one and several
workgroups along K, the padding prologue (K or N not a multiple of 8) and
misaligned operands at run time (which run the direct-to-LDS split-K plan's
own fallbacks). AddMM and fp16 inputs take the same kernels.
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


def note(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def device():
    torch()
    ac.adaptcore_init()
    yield


def offchip_candidates(M, N, K, dtype, limit=None):
    c = [x for x in all_candidates(M, N, K, dtype) if x["family_name"] == "offchip"]
    return c if limit is None else c[:limit]


def split_k_twin(key):
    """The direct-to-LDS split-K key with the same configuration and slices."""
    cfg = (key >> 4) & 0xF
    return (key & ~0x3FFF) | ac.AC_FAMILY_DL | (cfg << 4)


SHAPES = [(1100, 600, 3000), (512, 512, 4096), (300, 700, 1000), (777, 300, 2049), (1536, 256, 8192)]


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_offchip_matches_split_k_and_oracle(shape, dtype):
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=7 * M + N + 3 * K)
    ref = gemm_ref.gemm(A, B)
    cands = offchip_candidates(M, N, K, dtype)
    assert cands, shape
    kinds = set()
    for c in cands:
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        names = ac.adaptcore_plan_kernels(plan)
        assert names[-2].startswith("k_dl_sc<") and names[-1].startswith("k_reduce<"), names
        info = ac.adaptcore_plan_info(plan)
        kinds.add("single" if info["grid_y"] == 1 else "hybrid")
        vals, ok = run(plan, A, B, M, N, K, dtype)
        check(vals, ok, A, B, dtype, ref=ref, label="%s %s" % (shape, c))
        twin = forced_plan(M, N, K, dtype, split_k_twin(c["variant_key"]))
        assert ac.adaptcore_plan_info(twin)["pk"] == info["pk"]
        v2, ok2 = run(twin, A, B, M, N, K, dtype)
        assert ok2 and np.array_equal(vals.view(np.uint64), v2.view(np.uint64)), (shape, c)
    note("offchip", shape, dtype, len(cands), sorted(kinds))
    assert kinds == {"single", "hybrid"}


def test_offchip_integer_inputs_exact():
    M, N, K = 700, 520, 3000
    A, B = gen.operands(M, N, K, seed=83, dist="int")
    exact = (np.rint(gemm_ref.decode(A)).astype(np.int64) @ np.rint(gemm_ref.decode(B)).astype(np.int64))
    for c in offchip_candidates(M, N, K, F32):
        vals, ok = run(forced_plan(M, N, K, F32, c["variant_key"]), A, B, M, N, K, F32)
        assert ok and np.array_equal(vals, exact.astype(np.float64)), c


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
def test_offchip_misaligned_operands(dtype):
    """An odd leading dimension or a 2-byte offset: the call runs the
    direct-to-LDS split-K plan with the same slices (its register-load form)
    and still matches the oracle."""
    M, N, K = 600, 520, 2048
    A, B = gen.operands(M, N, K, seed=89)
    ref = gemm_ref.gemm(A, B)
    for c in offchip_candidates(M, N, K, dtype, limit=6):
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        for kw in [dict(lda=K + 3), dict(a_off=1), dict(ldb=N + 5)]:
            vals, ok = run(plan, A, B, M, N, K, dtype, **kw)
            check(vals, ok, A, B, dtype, ref=ref, label="%s %s" % (kw, c))


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
def test_offchip_addmm(dtype):
    M, N, K = 900, 600, 1500
    A, B = gen.operands(M, N, K, seed=97)
    old32 = gen.uniform_f32(M, N, 98)
    old = old32 if dtype == F32 else gen.bf16_bits(old32)
    old_vals = old32.astype(np.float64) if dtype == F32 else gemm_ref.decode(old)
    bias = gen.uniform_f32(1, N, 99).reshape(-1)
    R, D = addmm_ref.addmm(A, B, old_vals, 0.5, -0.25, bias)
    for c in offchip_candidates(M, N, K, dtype, limit=6):
        vals, ok = run_addmm(forced_plan(M, N, K, dtype, c["variant_key"]), A, B, M, N, K, dtype, old, 0.5, -0.25,
                             bias)
        assert ok, c
        assert gemm_ref.err_metric(vals, R, D) <= tol(dtype), c


@pytest.mark.parametrize("dtype", [ac.AC_F16_F32OUT, ac.AC_F16_F16OUT], ids=["f32out", "f16out"])
def test_offchip_fp16(dtype):
    M, N, K = 800, 512, 2000
    A, B = gen.operands(M, N, K, seed=101, dist="uniform_f16")
    ref = gemm_ref.gemm(A, B, fmt="fp16")
    for c in offchip_candidates(M, N, K, dtype, limit=6):
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        assert "f16::k_dl_sc<" in ";".join(ac.adaptcore_plan_kernels(plan))
        vals, ok = run(plan, A, B, M, N, K, dtype)
        check(vals, ok, A, B, dtype, ref=ref, label=str(c))
