"""GPU parity: every kernel configuration against the fp64 oracle.

Each case runs through the C ABI (adaptcore_plan / adaptcore_plan_variant +
adaptcore_matmul) on bf16 inputs and compares element by element with
oracle.gemm_ref:  max_ij |C - C_ref| / sum_k |A_ik B_kj|  <= 1e-3 (fp32
output) or 8e-3 (bf16 output). Inputs whose partial sums are exact in fp32
give bitwise checks of every split and fix-up path. Output buffers carry
canaries around C to catch writes out of bounds.
"""
import sys

import numpy as np
import pytest

import paper_2608_10803_amd as ac
from oracle import gemm_ref
from workloads import gen

from gpu_util import all_candidates, check, forced_plan, run, torch

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


def test_single_512_default_plan():
    M = N = K = 512
    A, B = gen.operands(M, N, K, seed=1)
    plan = ac.adaptcore_plan(M, N, K, F32)
    note("512^3", ac.adaptcore_plan_info(plan))
    vals, ok = run(plan, A, B, M, N, K, F32)
    check(vals, ok, A, B, F32)


SMALL = [(1, 1, 1), (7, 5, 3), (16, 16, 16), (17, 33, 65), (33, 17, 129), (64, 64, 64),
         (65, 127, 200), (128, 128, 128), (129, 255, 257), (200, 300, 1000), (255, 64, 1),
         (1, 300, 777), (3, 1000, 100), (500, 7, 300), (256, 256, 512), (40, 9, 2000),
         (300, 600, 70), (1000, 20, 33)]


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "x".join(map(str, s)))
def test_every_configuration(shape, dtype):
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=M * 7 + N * 3 + K)
    ref = gemm_ref.gemm(A, B)
    cands = all_candidates(M, N, K, dtype)
    assert cands
    note("shape", shape, "dtype", dtype, "configurations", len(cands))
    fams = set()
    for c in cands:
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        vals, ok = run(plan, A, B, M, N, K, dtype)
        check(vals, ok, A, B, dtype, ref=ref, label="%s %s" % (shape, c))
        fams.add(c["family_name"])
    note("  families", sorted(fams))


INT_SHAPES = [(100, 200, 3000), (16, 5000, 4096), (3000, 8, 2000), (64, 64, 4096), (5, 77, 999)]


@pytest.mark.parametrize("shape", INT_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_integer_inputs_exact_for_every_configuration(shape):
    """Integer inputs in [-4, 4]: every partial sum is exact in fp32, so every
    split, reduction and fix-up order must give the exact integer product."""
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=11, dist="int")
    exact = (np.rint(gemm_ref.decode(A)).astype(np.int64) @ np.rint(gemm_ref.decode(B)).astype(np.int64))
    cands = all_candidates(M, N, K, F32)
    note("int", shape, len(cands))
    for c in cands:
        plan = forced_plan(M, N, K, F32, c["variant_key"])
        vals, ok = run(plan, A, B, M, N, K, F32)
        assert ok, c
        assert np.array_equal(vals, exact.astype(np.float64)), c


def test_split_paths_are_deterministic():
    M, N, K = 96, 160, 20000
    A, B = gen.operands(M, N, K, seed=21)
    for c in all_candidates(M, N, K, F32):
        if c["pk"] <= 1 and c["family_name"] != "streamk":
            continue
        plan = forced_plan(M, N, K, F32, c["variant_key"])
        v1, ok1 = run(plan, A, B, M, N, K, F32)
        v2, ok2 = run(plan, A, B, M, N, K, F32)
        assert ok1 and ok2 and np.array_equal(v1, v2), c


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
def test_identity_and_ones(dtype):
    M, K = 77, 300
    A = gen.uniform_bf16(M, K, 31)
    I = gen.bf16_bits(np.eye(K, dtype=np.float32))
    for c in all_candidates(M, K, K, dtype)[:40]:
        vals, ok = run(forced_plan(M, K, K, dtype, c["variant_key"]), A, I, M, K, K, dtype)
        assert ok and np.array_equal(vals, gemm_ref.decode(A)), c
    K = 4000
    A = gen.bf16_bits(np.ones((50, K), np.float32))
    B = gen.bf16_bits(np.ones((K, 60), np.float32))
    want = float(gemm_ref.decode(gen.bf16_bits(np.array([K], np.float32)))[0]) if dtype == BF16 else float(K)
    for c in all_candidates(50, 60, K, dtype):
        vals, ok = run(forced_plan(50, 60, K, dtype, c["variant_key"]), A, B, 50, 60, K, dtype)
        assert ok and np.all(vals == want), c


def test_transposition():
    M, N, K = 123, 45, 678
    A, B = gen.operands(M, N, K, seed=41)
    v1, ok1 = run(ac.adaptcore_plan(M, N, K, F32), A, B, M, N, K, F32)
    At, Bt = np.ascontiguousarray(B.T), np.ascontiguousarray(A.T)
    v2, ok2 = run(ac.adaptcore_plan(N, M, K, F32), At, Bt, N, M, K, F32)
    C_ref, D = gemm_ref.gemm(A, B)
    assert ok1 and ok2
    assert gemm_ref.err_metric(v1, C_ref, D) <= 1e-3
    assert gemm_ref.err_metric(v2.T, C_ref, D) <= 1e-3


def test_degenerate_dimensions():
    # K = 0: C is set to zero (the canary-filled output is overwritten)
    for M, N in [(5, 7), (300, 200)]:
        A = np.zeros((M, 0), np.uint16)
        B = np.zeros((0, N), np.uint16)
        for dt in (F32, BF16):
            vals, ok = run(ac.adaptcore_plan(M, N, 0, dt), A, B, M, N, 0, dt, lda=1)
            assert ok and np.all(vals == 0)
    # M = 0 or N = 0: nothing is written
    A, B = gen.operands(0, 9, 5, seed=1)
    vals, ok = run(ac.adaptcore_plan(0, 9, 5, F32), A, B, 0, 9, 5, F32)
    assert ok and vals.shape == (0, 9)
    A, B = gen.operands(4, 0, 5, seed=1)
    vals, ok = run(ac.adaptcore_plan(4, 0, 5, F32), A, B, 4, 0, 5, F32, ldb=1, ldc=1)
    assert ok


@pytest.mark.parametrize("shape", [(37, 91, 333), (5, 4000, 1000), (2000, 12, 500), (300, 300, 3000)],
                         ids=lambda s: "x".join(map(str, s)))
def test_padded_leading_dimensions_and_unaligned_pointers(shape):
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=51)
    ref = gemm_ref.gemm(A, B)
    for c in all_candidates(M, N, K, BF16)[:30]:
        plan = forced_plan(M, N, K, BF16, c["variant_key"])
        vals, ok = run(plan, A, B, M, N, K, BF16, lda=K + 3, ldb=N + 5, ldc=N + 1, a_off=1, b_off=3)
        check(vals, ok, A, B, BF16, ref=ref, label=str(c))


def test_workspace_reuse_across_plans_and_streams():
    """Split-K counters are left at zero by every kernel, so plans of different
    shapes can share a stream's workspace; a second stream has its own."""
    t = torch()
    s2 = t.cuda.Stream()
    shapes = [(64, 64, 65536), (16, 4096, 4096), (512, 512, 20000), (3000, 8, 5000), (64, 64, 65536)]
    for i, (M, N, K) in enumerate(shapes):
        A, B = gen.operands(M, N, K, seed=60 + i, dist="int")
        exact = (np.rint(gemm_ref.decode(A)).astype(np.int64) @ np.rint(gemm_ref.decode(B)).astype(np.int64))
        for stream in (0, s2.cuda_stream):
            vals, ok = run(ac.adaptcore_plan(M, N, K, F32), A, B, M, N, K, F32, stream=stream)
            assert ok and np.array_equal(vals, exact.astype(np.float64)), (M, N, K)


@pytest.mark.parametrize("shape", [(4096, 2048, 40), (3000, 2000, 64), (1500, 1300, 130)],
                         ids=lambda s: "x".join(map(str, s)))
def test_persistent_streamk_configurations(shape):
    """Stream-K with more tiles than persistent workgroups, including the
    pure data-parallel form (one k-block per tile, or a whole number of
    waves), against the oracle."""
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=M + N + K)
    ref = gemm_ref.gemm(A, B)
    cands = [c for c in all_candidates(M, N, K, BF16) if c["family_name"] == "streamk"]
    assert cands
    for c in cands:
        plan = forced_plan(M, N, K, BF16, c["variant_key"])
        vals, ok = run(plan, A, B, M, N, K, BF16)
        check(vals, ok, A, B, BF16, ref=ref, label="%s %s" % (shape, c))


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
@pytest.mark.parametrize("shape", [(4200, 4200, 72), (2100, 3000, 200), (3001, 2999, 129)],
                         ids=lambda s: "x".join(map(str, s)))
def test_persistent_tile_configurations(shape, dtype):
    """The persistent tile kernels (more tiles than workgroups, the next
    tile's first k-block fetched before the epilogue) against the oracle, and
    bitwise equal to the depth-1 tile kernel of the same tile and order (the
    same k-order for every output)."""
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=M + N + K + 5)
    ref = gemm_ref.gemm(A, B)
    cands = all_candidates(M, N, K, dtype)
    pers = [c for c in cands if c["family_name"] == "persist"]
    assert pers
    twins = {}
    for c in cands:
        if c["family_name"] == "tile" and c["pk"] == 1:
            name = ac.adaptcore_plan_kernels(forced_plan(M, N, K, dtype, c["variant_key"]))[0]
            if name.endswith(", 1>"):  # depth 1
                twins[(c["tile_m"], c["tile_n"], (c["variant_key"] >> 12) & 1)] = c["variant_key"]
    for c in pers:
        note("persistent", shape, c["tile_m"], c["tile_n"], hex(c["variant_key"]))
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        vals, ok = run(plan, A, B, M, N, K, dtype)
        check(vals, ok, A, B, dtype, ref=ref, label="%s %s" % (shape, c))
        key = twins.get((c["tile_m"], c["tile_n"], (c["variant_key"] >> 12) & 1))
        if key is not None:
            vt, ok2 = run(forced_plan(M, N, K, dtype, key), A, B, M, N, K, dtype)
            assert ok2 and np.array_equal(vt, vals), "persistent differs from the tile kernel %s" % c



# ---- fp16 inputs (the same kernels built for the fp16 MFMA instructions)

SMALL_F16 = [(1, 1, 1), (7, 5, 3), (17, 33, 65), (129, 255, 257), (200, 300, 1000), (255, 64, 1),
             (3, 1000, 100), (500, 7, 300), (300, 600, 70), (1000, 20, 33)]


@pytest.mark.parametrize("dtype", [F16F32, F16F16], ids=["f16_f32out", "f16_f16out"])
@pytest.mark.parametrize("shape", SMALL_F16, ids=lambda s: "x".join(map(str, s)))
def test_fp16_every_configuration(shape, dtype):
    M, N, K = shape
    A, B = gen.operands(M, N, K, seed=M * 5 + N * 3 + K, dist="uniform_f16")
    ref = gemm_ref.gemm(A, B, fmt="fp16")
    cands = all_candidates(M, N, K, dtype)
    assert cands
    note("fp16 shape", shape, "dtype", dtype, "configurations", len(cands))
    for c in cands:
        plan = forced_plan(M, N, K, dtype, c["variant_key"])
        # the kernels of the fp16 build (the prologue copies move 16-bit
        # patterns and are shared by both formats)
        names = ac.adaptcore_plan_kernels(plan)
        assert all(k.startswith("f16::") for k in names if k not in ("k_pad16", "k_transpose16")), names
        vals, ok = run(plan, A, B, M, N, K, dtype)
        check(vals, ok, A, B, dtype, ref=ref, label="%s %s" % (shape, c))


@pytest.mark.parametrize("dtype", [F16F32, F16F16], ids=["f16_f32out", "f16_f16out"])
def test_fp16_default_plans_and_persistent(dtype):
    """Default plans of larger shapes and every persistent configuration of
    one shape with more tiles than workgroups, fp16 inputs."""
    for (M, N, K) in [(2100, 3000, 200), (640, 1000, 4096), (4, 4096, 4096)]:
        A, B = gen.operands(M, N, K, seed=M + N + K, dist="uniform_f16")
        ref = gemm_ref.gemm(A, B, fmt="fp16")
        keys = [ac.adaptcore_plan_info(ac.adaptcore_plan(M, N, K, dtype))["variant_key"]]
        if (M, N, K) == (2100, 3000, 200):
            keys += [c["variant_key"] for c in all_candidates(M, N, K, dtype) if c["family_name"] == "persist"]
        for k in keys:
            plan = forced_plan(M, N, K, dtype, k)
            note("fp16", (M, N, K), ac.adaptcore_plan_kernels(plan))
            vals, ok = run(plan, A, B, M, N, K, dtype)
            check(vals, ok, A, B, dtype, ref=ref, label="%s %s" % ((M, N, K), hex(k)))


def test_plan_before_init_equals_plan_after_init():
    """The planner prices candidates with the occupancies the device reports
    whatever the order of the first calls: in a fresh process, plans made
    before adaptcore_init equal those made after it (cache cleared)."""
    import json
    import subprocess
    import sys
    code = r'''
import json, paper_2608_10803_amd as ac
shapes = [(64, 64, 20000), (3000, 5, 700), (33, 4096, 4096), (700, 900, 3000), (16, 16, 16), (2048, 2048, 2048)]
first = [ac.adaptcore_plan_info(ac.adaptcore_plan(*s, 0))["variant_key"] for s in shapes]
ac.adaptcore_init()
ac.adaptcore_cache_clear()
second = [ac.adaptcore_plan_info(ac.adaptcore_plan(*s, 0))["variant_key"] for s in shapes]
print(json.dumps([first, second]))
'''
    root = __import__("os").path.dirname(__import__("os").path.dirname(__import__("os").path.abspath(__file__)))
    out = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr[-2000:]
    first, second = json.loads(out.stdout.strip().splitlines()[-1])
    assert first == second
