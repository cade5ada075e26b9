"""Calls captured in a HIP graph and replayed.

The benchmark times graph replays, and callers capture the library's calls
too: a plain plan, a split-K plan (partials in the stream's workspace), a
plan with a column-major B (the prologue copy in the workspace), AddMM with
beta != 0, a grouped product and a strided batch are captured on one stream
(workspace reserved beforehand: no allocation under capture) and replayed
three times, with the program's own eager work between the replays (inputs
of AddMM restored, every output overwritten with NaN); every replay is
checked against the oracle.
"""
import numpy as np
import pytest

import paper_2608_10803_amd as ac
from oracle import addmm_ref, gemm_ref, grouped_ref, layout_ref
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


def test_graph_replays_match_the_oracle():
    t = torch()
    ac.adaptcore_init()
    s = t.cuda.Stream()
    ac.adaptcore_reserve_workspace(s.cuda_stream, 256 << 20)
    calls, checks = [], []

    # plain and split-K plans
    for (M, N, K, dtype) in [(300, 600, 700, BF16), (64, 64, 20000, F32)]:
        A, B = gen.operands(M, N, K, seed=M + K)
        Ad, Bd = _dev(A), _dev(B)
        C = t.empty(M, N, dtype=t.float32 if dtype == F32 else t.bfloat16, device="cuda")
        plan = ac.adaptcore_plan(M, N, K, dtype)
        calls.append(lambda plan=plan, Ad=Ad, Bd=Bd, C=C, K=K, N=N: ac.adaptcore_matmul(
            plan, Ad.data_ptr(), K, Bd.data_ptr(), N, C.data_ptr(), N, s.cuda_stream))
        checks.append((C, dtype, gemm_ref.gemm(A, B), None, (Ad, Bd)))
    assert ac.adaptcore_plan_info(ac.adaptcore_plan(64, 64, 20000, F32))["pk"] > 1

    # column-major B (prologue copy into the workspace)
    M, N, K = 200, 300, 400
    A, B = gen.operands(M, N, K, seed=5)
    Bt = np.ascontiguousarray(B.T)
    Ad, Bd = _dev(A), _dev(Bt)
    C = t.empty(M, N, dtype=t.float32, device="cuda")
    plan = ac.adaptcore_plan(M, N, K, F32, ac.AC_LAYOUT_B_COL)
    assert "k_transpose16" in ac.adaptcore_plan_kernels(plan)
    calls.append(lambda plan=plan, Ad=Ad, Bd=Bd, C=C: ac.adaptcore_matmul(
        plan, Ad.data_ptr(), 400, Bd.data_ptr(), 400, C.data_ptr(), 300, s.cuda_stream))
    checks.append((C, F32, layout_ref.gemm_layout(A.reshape(-1), Bt.reshape(-1), M, N, K, K, K, 2), None, (Ad, Bd)))

    # AddMM with beta != 0: C is restored before every replay
    M, N, K = 150, 260, 330
    A, B = gen.operands(M, N, K, seed=6)
    old = gen.uniform_f32(M, N, 7)
    bias = gen.uniform_f32(1, N, 8).reshape(-1)
    Ad, Bd, biasd = _dev(A), _dev(B), t.from_numpy(bias).cuda()
    C0 = t.from_numpy(old).cuda()
    C = C0.clone()
    plan = ac.adaptcore_plan(M, N, K, F32)
    calls.append(lambda plan=plan, Ad=Ad, Bd=Bd, C=C: ac.adaptcore_addmm(
        plan, Ad.data_ptr(), 330, Bd.data_ptr(), 260, C.data_ptr(), 260, 0.5, -1.5, biasd.data_ptr(), s.cuda_stream))
    checks.append((C, F32, addmm_ref.addmm(A, B, old.astype(np.float64), 0.5, -1.5, bias), C0, (Ad, Bd, biasd)))

    # grouped product (device counts) and strided batch
    counts = np.array([40, 0, 75], np.int32)
    rows, N, K = 130, 96, 200
    A = gen.uniform_bf16(rows, K, 9)
    B = np.concatenate([gen.uniform_bf16(K, N, 10 + g).reshape(-1) for g in range(3)])
    Ad, Bd, cnt = _dev(A), _dev(B), t.from_numpy(counts).cuda()
    Cg = t.empty(rows, N, dtype=t.float32, device="cuda")
    gplan = ac.adaptcore_grouped_plan(rows, 3, N, K, F32)
    calls.append(lambda: ac.adaptcore_grouped_matmul(gplan, cnt.data_ptr(), Ad.data_ptr(), K, Bd.data_ptr(), N, K * N,
                                                     Cg.data_ptr(), N, s.cuda_stream))
    gref = grouped_ref.grouped_gemm(A, B, counts, rows, N, K, K, N, K * N)
    batch, Mb = 3, 40
    Ab = gen.uniform_bf16(batch * Mb, K, 11)
    Abd = _dev(Ab)
    Cb = t.empty(batch * Mb, N, dtype=t.float32, device="cuda")
    bplan = ac.adaptcore_batched_plan(batch, Mb, N, K, F32)
    calls.append(lambda: ac.adaptcore_batched_matmul(bplan, Abd.data_ptr(), K, Mb * K, Bd.data_ptr(), N, K * N,
                                                     Cb.data_ptr(), N, Mb * N, s.cuda_stream))
    bref = grouped_ref.batched_gemm(Ab.reshape(-1), B, batch, Mb, N, K, K, N, Mb * K, K * N)

    g = t.cuda.CUDAGraph()
    with t.cuda.graph(g, stream=s):
        for call in calls:
            call()
    for replay in range(3):
        # the program's own eager work between replays
        for (C, _, _, restore, _) in checks:
            if restore is not None:
                C.copy_(restore)
            else:
                C.fill_(float("nan"))
        Cg.fill_(float("nan"))
        Cb.fill_(float("nan"))
        t.cuda.synchronize()
        g.replay()
        t.cuda.synchronize()
        for i, (C, dtype, (R, D), _, _) in enumerate(checks):
            err = gemm_ref.err_metric(_vals(C, dtype), R, D)
            assert err <= tol(dtype), (replay, i, err)
        R, D, cov = gref
        got = Cg.cpu().numpy().astype(np.float64)
        assert gemm_ref.err_metric(got[cov], R[cov], D[cov]) <= tol(F32), replay
        R, D = bref
        got = Cb.cpu().numpy().astype(np.float64)
        assert gemm_ref.err_metric(got, R.reshape(-1, N), D.reshape(-1, N)) <= tol(F32), replay


def test_capture_without_workspace_is_an_error():
    """A split-K plan whose workspace (512 MiB) is larger than any other test
    reserves, captured on a stream: the call refuses to allocate under
    capture and reports AC_ERR_NOT_INITIALIZED (the operands are real
    buffers of the full size all the same)."""
    t = torch()
    ac.adaptcore_init()
    s = t.cuda.Stream()
    M, N, K = 2048, 2048, 131072
    keys = [c["variant_key"] for c in all_candidates(M, N, K, F32)
            if c["family_name"] == "tile" and c["pk"] == 32 and c["tile_m"] == 256 and c["tile_n"] == 256]
    assert keys
    plan = forced_plan(M, N, K, F32, keys[0])
    assert ac.adaptcore_plan_info(plan)["workspace_bytes"] >= 512 << 20
    Ad = t.empty(M * K, dtype=t.bfloat16, device="cuda")
    Bd = t.empty(K * N, dtype=t.bfloat16, device="cuda")
    C = t.empty(M, N, dtype=t.float32, device="cuda")
    g = t.cuda.CUDAGraph()
    status = None
    with t.cuda.graph(g, stream=s):
        try:
            ac.adaptcore_matmul(plan, Ad.data_ptr(), K, Bd.data_ptr(), N, C.data_ptr(), N, s.cuda_stream)
        except ac.AdaptCoreError as e:
            status = e.status
        C.fill_(0.0)  # something to capture
    assert status == ac.AC_ERR_NOT_INITIALIZED


def test_workspace_growth_after_capture_keeps_the_captured_buffer():
    """A split-K call captured on a stream with a small reserved workspace,
    then an eager call on the same stream whose plan needs a larger one (the
    workspace grows), then new device allocations filled with a pattern, then
    replays of the graph: the captured call keeps using its buffer, which the
    growth retired but did not free. Every replay matches the oracle, and
    the buffers allocated after the growth keep their pattern."""
    t = torch()
    ac.adaptcore_init()
    s = t.cuda.Stream()
    M, N, K = 64, 64, 20000
    small = ac.adaptcore_plan(M, N, K, F32)
    ws_small = ac.adaptcore_plan_info(small)["workspace_bytes"]
    assert ac.adaptcore_plan_info(small)["pk"] > 1 and ws_small > 0
    ac.adaptcore_reserve_workspace(s.cuda_stream, ws_small)
    A, B = gen.operands(M, N, K, seed=21)
    Ad, Bd = _dev(A), _dev(B)
    C = t.empty(M, N, dtype=t.float32, device="cuda")
    g = t.cuda.CUDAGraph()
    with t.cuda.graph(g, stream=s):
        ac.adaptcore_matmul(small, Ad.data_ptr(), K, Bd.data_ptr(), N, C.data_ptr(), N, s.cuda_stream)
    # an eager split-K call that needs a workspace larger than the reserved one
    M2, N2, K2 = 512, 512, 65536
    keys = [c["variant_key"] for c in all_candidates(M2, N2, K2, F32)
            if c["family_name"] == "tile" and c["pk"] >= 16]
    assert keys
    big = forced_plan(M2, N2, K2, F32, keys[0])
    assert ac.adaptcore_plan_info(big)["workspace_bytes"] > 4 * max(ws_small, 1 << 20)
    A2, B2 = gen.operands(M2, N2, 512, seed=22)  # K2 rows built from a tiled 512-deep slice
    A2 = np.tile(A2, (1, K2 // 512))
    B2 = np.tile(B2, (K2 // 512, 1))
    A2d, B2d = _dev(A2), _dev(B2)
    C2 = t.empty(M2, N2, dtype=t.float32, device="cuda")
    with t.cuda.stream(s):
        ac.adaptcore_matmul(big, A2d.data_ptr(), K2, B2d.data_ptr(), N2, C2.data_ptr(), N2, s.cuda_stream)
    s.synchronize()
    rows = np.arange(0, M2, 37)
    R2, D2 = gemm_ref.gemm(A2[rows], B2)
    assert gemm_ref.err_metric(C2.cpu().numpy().astype(np.float64)[rows], R2, D2) <= tol(F32)
    # allocations made after the growth: a freed buffer would be handed out here
    fillers = [t.full((max(ws_small, 1 << 20) // 4 + 64,), 7.0, device="cuda") for _ in range(4)]
    ref = gemm_ref.gemm(A, B)
    for replay in range(3):
        C.fill_(float("nan"))
        t.cuda.synchronize()
        g.replay()
        t.cuda.synchronize()
        assert gemm_ref.err_metric(C.cpu().numpy().astype(np.float64), *ref) <= tol(F32), replay
        assert all(bool((f == 7.0).all()) for f in fillers), replay
