"""Parity at the full workload sizes, in the configuration the benchmark runs
(the planner's own choice for each shape, packed row-major operands).

The outputs are too large for the oracle to compute whole, so each shape is
checked on sampled entries: the four corners, the last rows and columns of
ragged tiles and a seeded random sample. The oracle computes those entries
one by one from the A rows and B columns they need, read back from the
device buffers the kernels consumed (the inputs come from torch's seeded
generator, never from this library). Bar: the error metric per entry,
|C - C_ref| / sum_k |A_ik B_kj|, within the tolerance of the output type.
"""
import math
import sys

import numpy as np
import pytest

import paper_2608_10803_amd as ac
from oracle import addmm_ref
from oracle import gemm_ref
from workloads import gen

from gpu_util import tol

pytestmark = pytest.mark.gpu

F32, BF16 = ac.AC_BF16_F32OUT, ac.AC_BF16_BF16OUT
N_RANDOM = 28


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a GPU")
    return torch


class Arena:
    """Device buffers large enough for every operand of a workload; operand
    values drawn once per buffer from a seeded generator."""

    def __init__(self, shapes, dtype, seed, dist="uniform"):
        t = _torch()
        self.t = t
        na = max(max(M * K for M, N, K in shapes), 1)
        nb = max(max(K * N for M, N, K in shapes), 1)
        nc = max(max(M * N for M, N, K in shapes), 1)
        g = t.Generator(device="cuda")
        g.manual_seed(seed)
        self.A = t.empty(na, dtype=t.bfloat16, device="cuda")
        self.B = t.empty(nb, dtype=t.bfloat16, device="cuda")
        if dist == "uniform":
            self.A.uniform_(-1, 1, generator=g)
            self.B.uniform_(-1, 1, generator=g)
        self.dist = dist
        self.g = g
        self.C = t.empty(nc, dtype=t.float32 if dtype == F32 else t.bfloat16, device="cuda")

    def fill_normal(self, M, N, K):
        s = 1.0 / math.sqrt(K)
        self.A[:M * K].normal_(0.0, s, generator=self.g)
        self.B[:K * N].normal_(0.0, s, generator=self.g)


def _tile_edges(L, tile, rng, most=12):
    """First and last index of up to `most` tiles of size `tile` along a
    dimension of L (always the last, possibly ragged, tile), in random order."""
    nt = (L + tile - 1) // tile
    ts = sorted(set(np.linspace(0, nt - 1, min(nt, most)).astype(np.int64).tolist()) | {nt - 1})
    idx = []
    for t in ts:
        idx += [t * tile, min((t + 1) * tile, L) - 1]
    return list(rng.permutation(np.array(idx, np.int64)))


def sample_entries(M, N, seed, tile_m=256, tile_n=256):
    """The four corners, the first and last row / column of tiles of the
    plan's own tiling (the last, ragged tile always) paired with random
    columns / rows, and N_RANDOM random entries."""
    rng = np.random.default_rng(seed)
    I = [0, M - 1, 0, M - 1]
    J = [0, N - 1, N - 1, 0]
    ei = _tile_edges(M, max(tile_m, 1), rng)
    ej = _tile_edges(N, max(tile_n, 1), rng)
    I += ei + list(rng.integers(0, M, len(ej)))
    J += list(rng.integers(0, N, len(ei))) + ej
    I += list(rng.integers(0, M, N_RANDOM))
    J += list(rng.integers(0, N, N_RANDOM))
    return np.array(I, np.int64), np.array(J, np.int64)


def assert_covered(t, C, label):
    """C was filled with NaN before the call and the inputs are finite: every
    entry must have been written."""
    assert not bool(t.isnan(C).any()), "%s: entries of C left unwritten" % (label,)


def check_shape(arena, M, N, K, dtype, seed, label):
    t = arena.t
    plan = ac.adaptcore_plan(M, N, K, dtype, 0)
    A = arena.A[:M * K].view(M, K) if K else arena.A[:0]
    B = arena.B[:K * N].view(K, N) if K else arena.B[:0]
    C = arena.C[:M * N].view(M, N)
    C.fill_(float("nan"))
    ac.adaptcore_matmul(plan, arena.A.data_ptr(), max(K, 1), arena.B.data_ptr(), max(N, 1),
                        arena.C.data_ptr(), max(N, 1), 0)
    t.cuda.synchronize()
    d = ac.adaptcore_plan_info(plan)
    assert_covered(t, C, "%s %s" % (label, (M, N, K)))
    I, J = sample_entries(M, N, seed, d["tile_m"], d["tile_n"])
    got = C[t.from_numpy(I).cuda(), t.from_numpy(J).cuda()]
    if dtype == F32:
        vals = got.cpu().numpy().astype(np.float64)
    else:
        vals = gemm_ref.decode(got.view(t.int16).cpu().numpy().view(np.uint16))
    # the A rows and B columns the sampled entries need, as raw bf16 bits
    ui, inv_i = np.unique(I, return_inverse=True)
    uj, inv_j = np.unique(J, return_inverse=True)
    Ar = A[t.from_numpy(ui).cuda()].contiguous().view(t.int16).cpu().numpy().view(np.uint16)
    Bc = B[:, t.from_numpy(uj).cuda()].contiguous().view(t.int16).cpu().numpy().view(np.uint16)
    C_ref, D = gemm_ref.gemm_entries(Ar, Bc, inv_i, inv_j, M=len(ui), N=len(uj), K=K)
    err = gemm_ref.err_metric(vals, C_ref, D)
    assert err <= tol(dtype), "%s %s err %.3g (%s %dx%d pk %d)" % (
        label, (M, N, K), err, d["family_name"], d["tile_m"], d["tile_n"], d["pk"])
    return err, d["family_name"]


def _progress(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def test_single_512_full_output():
    """The 512^3 case with fp32 output: every entry against the oracle."""
    t = _torch()
    (M, N, K), = gen.single_512()
    A, B = gen.operands(M, N, K, seed=1)
    C_ref, D = gemm_ref.gemm(A, B)
    plan = ac.adaptcore_plan(M, N, K, F32, 0)
    Ad = t.from_numpy(A.view(np.int16)).cuda()
    Bd = t.from_numpy(B.view(np.int16)).cuda()
    Cd = t.full((M, N), float("nan"), dtype=t.float32, device="cuda")
    ac.adaptcore_matmul(plan, Ad.data_ptr(), K, Bd.data_ptr(), N, Cd.data_ptr(), N, 0)
    t.cuda.synchronize()
    err = gemm_ref.err_metric(Cd.cpu().numpy().astype(np.float64), C_ref, D)
    assert err <= tol(F32), err


def test_skinny_m_full_size():
    shapes = gen.skinny_m()
    arena = Arena(shapes, BF16, seed=2)
    for i, (M, N, K) in enumerate(shapes):
        _progress("skinny %s" % ((M, N, K),))
        check_shape(arena, M, N, K, BF16, 100 + i, "skinny-M")


def test_small_mn_large_k_full_size():
    shapes = gen.small_mn_large_k()
    arena = Arena(shapes, F32, seed=3, dist="normal")
    for i, (M, N, K) in enumerate(shapes):
        _progress("split-K %s" % ((M, N, K),))
        arena.fill_normal(M, N, K)
        check_shape(arena, M, N, K, F32, 200 + i, "small-MN large-K")


def test_sweep_full_size():
    """Every shape of the 2,000-shape sweep, each with its planned
    configuration, on sampled entries."""
    shapes = gen.sweep()
    arena = Arena(shapes, BF16, seed=4)
    fams = {}
    for i, (M, N, K) in enumerate(shapes):
        if i % 250 == 0:
            _progress("sweep %d/%d" % (i, len(shapes)))
        _, f = check_shape(arena, M, N, K, BF16, 1000 + i, "sweep #%d" % i)
        fams[f] = fams.get(f, 0) + 1
    _progress("sweep families %s" % fams)


def test_moe_stream_full_size():
    """Two routing steps of the MoE stream: every expert's up- and
    down-projection (including experts with no tokens)."""
    shapes = []
    for counts in gen.moe_counts(steps=2):
        shapes += [(M, N, K) for (_, _, M, N, K) in gen.moe_shapes(counts)]
    arena = Arena([s for s in shapes if s[0] > 0] or [(1, 1, 1)], BF16, seed=5)
    for i, (M, N, K) in enumerate(shapes):
        if M == 0:
            plan = ac.adaptcore_plan(M, N, K, BF16, 0)
            ac.adaptcore_matmul(plan, arena.A.data_ptr(), K, arena.B.data_ptr(), N, arena.C.data_ptr(), N, 0)
            continue
        check_shape(arena, M, N, K, BF16, 5000 + i, "moe #%d" % i)


# the shapes of the benchmark's layouts workload
LAYOUT_SHAPES = [(4096, 4096, 4096), (2048, 14336, 4096), (8192, 8192, 1024), (16, 4096, 14336), (512, 512, 512)]


def _sampled(t, Alog, Blog, M, N, K, seed, plan=None):
    """Sampled entries and the raw bf16 A rows and B columns they need,
    read through the logical (possibly transposed) views."""
    d = ac.adaptcore_plan_info(plan) if plan is not None else {"tile_m": 256, "tile_n": 256}
    I, J = sample_entries(M, N, seed, d["tile_m"], d["tile_n"])
    ui, inv_i = np.unique(I, return_inverse=True)
    uj, inv_j = np.unique(J, return_inverse=True)
    Ar = Alog[t.from_numpy(ui).cuda()].contiguous().view(t.int16).cpu().numpy().view(np.uint16)
    Bc = Blog[:, t.from_numpy(uj).cuda()].contiguous().view(t.int16).cpu().numpy().view(np.uint16)
    return I, J, Ar, Bc, inv_i, inv_j, len(ui), len(uj)


def test_layouts_full_size():
    """The benchmark's layouts workload: each shape with A, B or both stored
    column-major, the planner's own plan, bf16 output, sampled entries."""
    t = _torch()
    g = t.Generator(device="cuda")
    g.manual_seed(6)
    for si, (M, N, K) in enumerate(LAYOUT_SHAPES):
        A = t.empty(M * K, dtype=t.bfloat16, device="cuda").uniform_(-1, 1, generator=g)
        B = t.empty(K * N, dtype=t.bfloat16, device="cuda").uniform_(-1, 1, generator=g)
        C = t.empty(M, N, dtype=t.bfloat16, device="cuda")
        for lay in (ac.AC_LAYOUT_A_COL, ac.AC_LAYOUT_B_COL, ac.AC_LAYOUT_COL_COL):
            a_col, b_col = bool(lay & 1), bool(lay & 2)
            _progress("layouts %d %s" % (lay, (M, N, K)))
            Alog = A.view(K, M).t() if a_col else A.view(M, K)
            Blog = B.view(N, K).t() if b_col else B.view(K, N)
            plan = ac.adaptcore_plan(M, N, K, BF16, lay)
            C.fill_(float("nan"))
            ac.adaptcore_matmul(plan, A.data_ptr(), M if a_col else K, B.data_ptr(), K if b_col else N,
                                C.data_ptr(), N, 0)
            t.cuda.synchronize()
            assert_covered(t, C, "layouts %d %s" % (lay, (M, N, K)))
            I, J, Ar, Bc, ii, jj, nu, nv = _sampled(t, Alog, Blog, M, N, K, 7000 + 10 * si + lay, plan)
            got = C[t.from_numpy(I).cuda(), t.from_numpy(J).cuda()]
            vals = gemm_ref.decode(got.view(t.int16).cpu().numpy().view(np.uint16))
            C_ref, D = gemm_ref.gemm_entries(Ar, Bc, ii, jj, M=nu, N=nv, K=K)
            err = gemm_ref.err_metric(vals, C_ref, D)
            assert err <= tol(BF16), ((M, N, K), lay, err, ac.adaptcore_plan_kernels(plan))


def test_addmm_full_size():
    """AddMM (alpha, beta, bias) at full size with fp32 and bf16 output, row-
    and column-major B, the planner's own plan, sampled entries."""
    t = _torch()
    g = t.Generator(device="cuda")
    g.manual_seed(8)
    for si, (M, N, K) in enumerate([(2048, 14336, 4096), (16, 4096, 14336), (8192, 8192, 1024)]):
        A = t.empty(M * K, dtype=t.bfloat16, device="cuda").uniform_(-1, 1, generator=g)
        B = t.empty(K * N, dtype=t.bfloat16, device="cuda").uniform_(-1, 1, generator=g)
        bias = t.empty(N, dtype=t.float32, device="cuda").uniform_(-1, 1, generator=g)
        for dtype in (F32, BF16):
            for lay in (0, ac.AC_LAYOUT_B_COL):
                _progress("addmm %s dtype %d layouts %d" % ((M, N, K), dtype, lay))
                C = t.empty(M, N, dtype=t.float32 if dtype == F32 else t.bfloat16, device="cuda")
                C.uniform_(-2, 2, generator=g)
                plan = ac.adaptcore_plan(M, N, K, dtype, lay)
                d = ac.adaptcore_plan_info(plan)
                I, J = sample_entries(M, N, 8000 + si, d["tile_m"], d["tile_n"])
                Ii, Jj = t.from_numpy(I).cuda(), t.from_numpy(J).cuda()
                old = C[Ii, Jj].float().cpu().numpy().astype(np.float64)
                Blog = B.view(N, K).t() if lay else B.view(K, N)
                ac.adaptcore_addmm(plan, A.data_ptr(), K, B.data_ptr(), K if lay else N, C.data_ptr(), N,
                                   0.75, -1.25, bias.data_ptr(), 0)
                t.cuda.synchronize()
                got = C[Ii, Jj]
                if dtype == F32:
                    vals = got.cpu().numpy().astype(np.float64)
                else:
                    vals = gemm_ref.decode(got.view(t.int16).cpu().numpy().view(np.uint16))
                _, _, Ar, Bc, ii, jj, nu, nv = _sampled(t, A.view(M, K), Blog, M, N, K, 8000 + si, plan)
                b = bias[Jj].cpu().numpy().astype(np.float64)
                C_ref, D = addmm_ref.addmm_entries(Ar, Bc, ii, jj, old, 0.75, -1.25, b, M=nu, N=nv, K=K)
                err = gemm_ref.err_metric(vals, C_ref, D)
                assert err <= tol(dtype), ((M, N, K), dtype, lay, err, ac.adaptcore_plan_kernels(plan))
