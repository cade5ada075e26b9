"""adaptcore_matmul_noalloc: the plain product with the library's fixed
device scratch as workspace, checked through the C ABI against
adaptcore_matmul (same plan, same kernels: equal bit for bit) and against
the oracle, on two calls in a row, the second with a smaller input; a
split-K plan, a column-major operand (prologue copy in the scratch), a plan
without workspace, and a plan whose workspace exceeds the scratch (refused,
nothing written)."""
import numpy as np
import pytest

import paper_2608_10803_amd as ac
from oracle import gemm_ref, layout_ref
from workloads import gen

from gpu_util import all_candidates, forced_plan, tol, torch

pytestmark = pytest.mark.gpu

F32, BF16 = ac.AC_BF16_F32OUT, ac.AC_BF16_BF16OUT


def _dev(bits):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


def _vals(C, dtype):
    if dtype == F32:
        return C.cpu().numpy().astype(np.float64)
    return gemm_ref.decode(C.view(torch().int16).cpu().numpy().view(np.uint16))


def _both(plan, Ad, lda, Bd, ldb, M, N, dtype, stream):
    """C from adaptcore_matmul_noalloc and from adaptcore_matmul (outputs
    pre-filled with NaN)."""
    t = torch()
    tdt = t.float32 if dtype == F32 else t.bfloat16
    C1 = t.full((M, N), float("nan"), dtype=tdt, device="cuda")
    C2 = t.full((M, N), float("nan"), dtype=tdt, device="cuda")
    ac.adaptcore_matmul_noalloc(plan, Ad.data_ptr(), lda, Bd.data_ptr(), ldb, C1.data_ptr(), N, stream)
    ac.adaptcore_matmul(plan, Ad.data_ptr(), lda, Bd.data_ptr(), ldb, C2.data_ptr(), N, stream)
    t.cuda.synchronize()
    return C1, C2


def _split_key(M, N, K, dtype, pk_min):
    """The tile configuration with the smallest split count >= pk_min."""
    keys = [c for c in all_candidates(M, N, K, dtype) if c["family_name"] == "tile" and c["pk"] >= pk_min]
    assert keys
    return min(keys, key=lambda c: (c["pk"], c["variant_key"]))["variant_key"]


def test_noalloc_matches_matmul_on_two_calls_second_smaller():
    t = torch()
    s = t.cuda.Stream()
    cap = ac.adaptcore_noalloc_scratch_bytes()
    assert cap == 64 << 20
    cases = [(512, 512, 16384, F32, 16), (96, 80, 5000, BF16, 4)]  # the second input is smaller
    for (M, N, K, dtype, pk_min) in cases:
        plan = forced_plan(M, N, K, dtype, _split_key(M, N, K, dtype, pk_min))
        d = ac.adaptcore_plan_info(plan)
        assert d["pk"] >= pk_min and 0 < d["workspace_bytes"] <= cap
        A, B = gen.operands(M, N, K, seed=M + N + K)
        Ad, Bd = _dev(A), _dev(B)
        C1, C2 = _both(plan, Ad, K, Bd, N, M, N, dtype, s.cuda_stream)
        v1, v2 = _vals(C1, dtype), _vals(C2, dtype)
        assert np.array_equal(v1.view(np.uint64), v2.view(np.uint64)), (M, N, K)
        R, D = gemm_ref.gemm(A, B)
        assert gemm_ref.err_metric(v1, R, D) <= tol(dtype), (M, N, K)


def test_noalloc_default_plans_and_column_major():
    t = torch()
    # the planner's own plans: a split-K shape, one without workspace, and a
    # column-major B (its row-major copy lives in the scratch); then a
    # smaller one of each again
    for (M, N, K, lay) in [(64, 64, 30000, 0), (700, 500, 300, 0), (300, 260, 900, ac.AC_LAYOUT_B_COL),
                           (33, 17, 4000, 0), (40, 30, 50, ac.AC_LAYOUT_B_COL)]:
        plan = ac.adaptcore_plan(M, N, K, F32, lay)
        A, B = gen.operands(M, N, K, seed=3 * M + K)
        if lay:
            Bs = np.ascontiguousarray(B.T)  # B stored column-major: N x K
            Ad, Bd = _dev(A), _dev(Bs)
            ldb = K
            R, D = layout_ref.gemm_layout(A.reshape(-1), Bs.reshape(-1), M, N, K, K, K, lay)
        else:
            Ad, Bd = _dev(A), _dev(B)
            ldb = N
            R, D = gemm_ref.gemm(A, B)
        C1, C2 = _both(plan, Ad, K, Bd, ldb, M, N, F32, 0)
        v1, v2 = _vals(C1, F32), _vals(C2, F32)
        assert np.array_equal(v1.view(np.uint64), v2.view(np.uint64)), (M, N, K, lay)
        assert gemm_ref.err_metric(v1, R, D) <= tol(F32), (M, N, K, lay)


def test_noalloc_refuses_a_workspace_beyond_the_scratch():
    t = torch()
    M, N, K = 2048, 2048, 65536
    key = _split_key(M, N, K, F32, 8)
    plan = forced_plan(M, N, K, F32, key)
    assert ac.adaptcore_plan_info(plan)["workspace_bytes"] > ac.adaptcore_noalloc_scratch_bytes()
    A = t.zeros(M * K, dtype=t.bfloat16, device="cuda")
    B = t.zeros(K * N, dtype=t.bfloat16, device="cuda")
    C = t.full((M, N), 3.0, dtype=t.float32, device="cuda")
    with pytest.raises(ac.AdaptCoreError) as e:
        ac.adaptcore_matmul_noalloc(plan, A.data_ptr(), K, B.data_ptr(), N, C.data_ptr(), N, 0)
    assert e.value.status == ac.AC_ERR_UNSUPPORTED
    t.cuda.synchronize()
    assert bool((C == 3.0).all())
