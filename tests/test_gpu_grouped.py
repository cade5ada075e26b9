"""GPU parity of the grouped product (adaptcore_grouped_matmul) against the
grouped oracle (oracle/grouped_ref.py).

Every grouped configuration runs on ragged sizes with padded leading
dimensions, empty groups and rows left uncovered; the counts live on the
device. Output buffers carry canaries: rows that no group covers, the row
above and below C and the columns past N must keep them. The MoE stream's
full-size steps (8192 tokens over 64 experts, both routing readings, up- and
down-projection) are checked on sampled entries. Bar: the error metric
max |C - C_ref| / sum_k |A_ik B_kj| within 1e-3 (fp32 out) or 8e-3 (bf16 out).
"""
import sys

import numpy as np
import pytest

import paper_2608_10803_amd as ac
from oracle import addmm_ref, gemm_ref, grouped_ref
from workloads import gen

from gpu_util import BF16_CANARY, F32_CANARY, Out, to_device, tol, torch

pytestmark = pytest.mark.gpu

F32, BF16 = ac.AC_BF16_F32OUT, ac.AC_BF16_BF16OUT


def note(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def device():
    torch()
    ac.adaptcore_init()
    yield


def grouped_keys(rows, G, N, K, dtype):
    """Every legal forced grouped configuration (both tile orders)."""
    keys = []
    for cfg in range(16):
        for sw in (0, 1):
            key = ac.AC_FAMILY_GROUPED | (cfg << 4) | (sw << 12) | (1 << 16) | (dtype << 48)
            try:
                ac.adaptcore_grouped_plan_variant(rows, G, N, K, dtype, 0, key)
            except ac.AdaptCoreError:
                continue
            keys.append(key)
    return keys


class Case:
    """Host operands of a grouped product: A (rows x K, lda), the groups' B
    matrices at multiples of stride_b (ldb), the counts."""

    def __init__(self, counts, rows, N, K, lda=None, ldb=None, stride_b=None, seed=0, shared_b=False):
        self.counts = np.asarray(counts, np.int32)
        self.G = len(counts)
        self.rows, self.N, self.K = rows, N, K
        self.lda = max(K, 1) if lda is None else lda
        self.ldb = max(N, 1) if ldb is None else ldb
        self.stride_b = (K * self.ldb if stride_b is None else stride_b) if not shared_b else 0
        self.A = gen.uniform_bf16(rows, K, seed) if rows and K else np.zeros((rows, K), np.uint16)
        nb = max(self.G - 1, 0) * self.stride_b + max(K - 1, 0) * self.ldb + N + 8
        self.B = np.zeros(nb, np.uint16)
        for g in range(self.G if not shared_b else 1):
            if K and N:
                m = gen.uniform_bf16(K, N, seed + 1 + g)
                view = np.lib.stride_tricks.as_strided(self.B[g * self.stride_b:], shape=(K, N),
                                                       strides=(self.ldb * 2, 2))
                view[...] = m

    def reference(self):
        Apad = np.zeros((self.rows, self.lda), np.uint16)
        Apad[:, :self.K] = self.A
        return grouped_ref.grouped_gemm(Apad, self.B, self.counts, self.rows, self.N, self.K, self.lda,
                                        self.ldb, self.stride_b)

    def run(self, plan, dtype, ldc=None, a_off=0):
        t = torch()
        ldc = max(self.N, 1) if ldc is None else ldc
        Ad, a = to_device(self.A, self.lda, a_off)
        Bd = t.from_numpy(self.B.view(np.int16)).to("cuda")
        cnt = t.from_numpy(self.counts).to("cuda")
        out = Out(self.rows, self.N, ldc, dtype)
        ac.adaptcore_grouped_matmul(plan, cnt.data_ptr(), a, self.lda, Bd.data_ptr(), self.ldb, self.stride_b,
                                    out.addr, ldc, 0)
        t.cuda.synchronize()
        vals, ok = out.read()
        raw = out.dev.cpu().numpy()
        if dtype == F32:
            body = raw.reshape(self.rows + 2, ldc)[1:self.rows + 1, :self.N]
            canary_rows = np.all(body == F32_CANARY, axis=1)
        else:
            body = raw.view(np.uint16).reshape(self.rows + 2, ldc)[1:self.rows + 1, :self.N]
            canary_rows = np.all(body == BF16_CANARY, axis=1)
        del Ad, Bd, cnt
        return vals, ok, canary_rows


    def run_addmm(self, plan, dtype, ldc, stored, alpha, beta, bias, stride_bias):
        """adaptcore_grouped_addmm with C holding `stored` (rows x N fp32
        values or 16-bit patterns); returns (values, canaries around C ok)."""
        t = torch()
        Ad, a = to_device(self.A, self.lda, 0)
        Bd = t.from_numpy(self.B.view(np.int16)).to("cuda")
        cnt = t.from_numpy(self.counts).to("cuda")
        bd = t.from_numpy(np.ascontiguousarray(bias, np.float32)).to("cuda")
        out = Out(self.rows, self.N, ldc, dtype)
        out.fill(stored)
        ac.adaptcore_grouped_addmm(plan, cnt.data_ptr(), a, self.lda, Bd.data_ptr(), self.ldb, self.stride_b,
                                   out.addr, ldc, alpha, beta, bd.data_ptr(), stride_bias, 0)
        t.cuda.synchronize()
        vals, ok = out.read()
        del Ad, Bd, cnt, bd
        return vals, ok


def check(case, vals, ok, canary_rows, dtype, ref, label):
    C_ref, D, cov = ref
    assert ok, "write outside C %s" % label
    assert np.all(canary_rows[~cov]), "a row no group covers was written %s" % label
    err = gemm_ref.err_metric(vals[cov], C_ref[cov], D[cov])
    assert err <= tol(dtype), "err %.3g > %.3g %s" % (err, tol(dtype), label)
    return err


RAGGED = dict(counts=[100, 0, 37, 250, 1, 0, 129, 64, 50], rows=700, N=300, K=197)


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
def test_every_grouped_configuration(dtype):
    c = RAGGED
    case = Case(c["counts"], c["rows"], c["N"], c["K"], lda=c["K"] + 5, ldb=c["N"] + 3,
                stride_b=c["K"] * (c["N"] + 3) + 11, seed=11)
    ref = case.reference()
    keys = grouped_keys(c["rows"], len(c["counts"]), c["N"], c["K"], dtype)
    assert len(keys) >= 10
    for key in keys:
        plan = ac.adaptcore_grouped_plan_variant(c["rows"], len(c["counts"]), c["N"], c["K"], dtype, 0, key)
        d = ac.adaptcore_plan_info(plan)
        label = "%s %dx%d sw%d" % (hex(key), d["tile_m"], d["tile_n"], d["swizzle"])
        note("grouped", label)
        vals, ok, canary = case.run(plan, dtype, ldc=c["N"] + 7)
        check(case, vals, ok, canary, dtype, ref, label)


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
def test_grouped_addmm_every_configuration(dtype):
    """The grouped product with the AddMM epilogue (a bias row per group) on
    every grouped configuration of the ragged case; rows no group covers
    keep their previous contents."""
    c = RAGGED
    rows, N, K, G = c["rows"], c["N"], c["K"], len(c["counts"])
    case = Case(c["counts"], rows, N, K, lda=K + 5, ldb=N + 3, stride_b=K * (N + 3) + 11, seed=12)
    if dtype == F32:
        stored = gen.uniform_f32(rows, N, 44, -2.0, 2.0)
        old = stored.astype(np.float64)
    else:
        stored = gen.uniform_bf16(rows, N, 44, -2.0, 2.0)
        old = gemm_ref.decode(stored)
    sbias = N + 9
    bias = gen.uniform_f32(1, (G - 1) * sbias + N, 45).reshape(-1)
    Apad = np.zeros((rows, K + 5), np.uint16)
    Apad[:, :K] = case.A
    C_ref, D, cov = addmm_ref.grouped_addmm(Apad, case.B, case.counts, rows, N, K, K + 5, N + 3, case.stride_b, old,
                                            1.25, -0.5, bias, sbias)
    for key in grouped_keys(rows, G, N, K, dtype):
        plan = ac.adaptcore_grouped_plan_variant(rows, G, N, K, dtype, 0, key)
        vals, ok = case.run_addmm(plan, dtype, N + 7, stored, 1.25, -0.5, bias, sbias)
        assert ok, "write outside C %s" % hex(key)
        assert np.array_equal(vals[~cov], old[~cov]), "an uncovered row changed %s" % hex(key)
        err = gemm_ref.err_metric(vals[cov], C_ref[cov], D[cov])
        assert err <= tol(dtype), "err %.3g %s" % (err, hex(key))


SHAPES = [
    # (counts, rows, N, K)
    ([3, 5, 0, 9], 17, 3, 5),                 # N < 8 and K < 8: the element-load path
    ([64, 128, 0, 256, 64], 512, 256, 256),   # whole tiles, aligned rows
    ([1] * 40, 40, 129, 64),                  # one row per group
    ([0, 0, 1000], 1000, 70, 1),              # K = 1
    ([300, 301], 700, 8, 1000),               # long K, narrow N
]


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "%dx%d_g%d" % (s[2], s[3], len(s[0])))
def test_default_plan_shapes(shape, dtype):
    counts, rows, N, K = shape
    case = Case(counts, rows, N, K, seed=rows + N + K)
    plan = ac.adaptcore_grouped_plan(rows, len(counts), N, K, dtype)
    note("grouped", shape, ac.adaptcore_plan_kernels(plan))
    vals, ok, canary = case.run(plan, dtype, a_off=1)
    check(case, vals, ok, canary, dtype, case.reference(), str(shape))


@pytest.mark.parametrize("sw", [0, 1])
def test_many_groups_scan_several_chunks(sw):
    """200 groups: the kernel's prefix scan spans four 64-group chunks."""
    rng = np.random.default_rng(5)
    w = rng.zipf(1.2, 200).astype(float)
    counts = rng.multinomial(3000, w / w.sum())
    rows, N, K = 3100, 130, 72
    case = Case(counts, rows, N, K, seed=7)
    ref = case.reference()
    for cfg in (3, 6):
        key = ac.AC_FAMILY_GROUPED | (cfg << 4) | (sw << 12) | (1 << 16) | (BF16 << 48)
        plan = ac.adaptcore_grouped_plan_variant(rows, 200, N, K, BF16, 0, key)
        vals, ok, canary = case.run(plan, BF16)
        check(case, vals, ok, canary, BF16, ref, "cfg %d sw %d" % (cfg, sw))


def test_negative_and_over_capacity_counts():
    """Negative counts read as 0; rows at or past the capacity are dropped."""
    counts = [50, -7, 80, 0, 200, 90]  # non-negative sum 420 > 300 rows
    case = Case(counts, 300, 96, 128, seed=9)
    ref = case.reference()
    assert ref[2].all()
    plan = ac.adaptcore_grouped_plan(300, len(counts), 96, 128, F32)
    vals, ok, canary = case.run(plan, F32)
    check(case, vals, ok, canary, F32, ref, "negative/over-capacity")


def test_shared_b_and_empty_cases():
    # stride_b = 0: every group multiplies by the same B
    case = Case([10, 0, 33, 70], 120, 40, 50, seed=13, shared_b=True)
    plan = ac.adaptcore_grouped_plan(120, 4, 40, 50, BF16)
    vals, ok, canary = case.run(plan, BF16)
    check(case, vals, ok, canary, BF16, case.reference(), "shared B")
    # all counts zero: nothing is written
    case = Case([0, 0, 0], 64, 32, 16, seed=14)
    vals, ok, canary = case.run(ac.adaptcore_grouped_plan(64, 3, 32, 16, F32), F32)
    assert ok and canary.all()
    # K = 0: covered rows become zero, the others keep their canaries
    case = Case([5, 0, 7], 20, 24, 0, seed=15)
    vals, ok, canary = case.run(ac.adaptcore_grouped_plan(20, 3, 24, 0, F32), F32)
    assert ok and np.all(vals[:12] == 0) and canary[12:].all() and not canary[:12].any()


def _sample_rows(counts, rows, rng, per_group=3):
    I = []
    for s, e in grouped_ref.group_rows(counts, rows):
        if e > s:
            I += [s, e - 1] + list(rng.integers(s, e, per_group))
    return np.array(I, np.int64)


@pytest.mark.parametrize("reading", ["B", "A"])
def test_moe_stream_full_size(reading):
    """Two routing steps of the MoE stream (8192 tokens, 64 experts): the
    up-projection (K 4096 -> N 1536) and down-projection (1536 -> 4096) of
    all experts, one grouped call each, checked on sampled entries."""
    t = torch()
    rows, G = 8192, 64
    for step, counts in enumerate(gen.moe_counts(steps=2, reading=reading)):
        for (N, K) in [(gen.MOE_FFN, gen.MOE_HIDDEN), (gen.MOE_HIDDEN, gen.MOE_FFN)]:
            note("moe", reading, step, (N, K))
            g = t.Generator(device="cuda")
            g.manual_seed(100 + step)
            A = t.empty(rows * K, dtype=t.bfloat16, device="cuda").uniform_(-1, 1, generator=g)
            B = t.empty(G * K * N, dtype=t.bfloat16, device="cuda").uniform_(-1, 1, generator=g)
            C = t.full((rows, N), float("nan"), dtype=t.bfloat16, device="cuda")
            cnt = t.from_numpy(np.asarray(counts, np.int32)).cuda()
            plan = ac.adaptcore_grouped_plan(rows, G, N, K, BF16)
            ac.adaptcore_grouped_matmul(plan, cnt.data_ptr(), A.data_ptr(), K, B.data_ptr(), N, K * N,
                                        C.data_ptr(), N, 0)
            t.cuda.synchronize()
            rng = np.random.default_rng(step)
            I = _sample_rows(counts, rows, rng)
            J = np.concatenate([[0, N - 1], rng.integers(0, N, len(I) - 2)])
            got = C[t.from_numpy(I).cuda(), t.from_numpy(J).cuda()]
            vals = gemm_ref.decode(got.view(t.int16).cpu().numpy().view(np.uint16))
            # the A rows and B columns the sampled entries need, as bf16 bits
            bounds = grouped_ref.group_rows(counts, rows)
            grp = np.array([next(k for k, (s, e) in enumerate(bounds) if s <= i < e) for i in I], np.int64)
            Ar = A.view(rows, K)[t.from_numpy(I).cuda()].view(t.int16).cpu().numpy().view(np.uint16)
            Bc = B.view(G, K, N)[t.from_numpy(grp).cuda(), :, t.from_numpy(J).cuda()]  # (samples, K)
            Bc = np.ascontiguousarray(Bc.view(t.int16).cpu().numpy().view(np.uint16).T)  # (K, samples)
            n = len(I)
            C_ref, D = gemm_ref.gemm_entries(Ar, Bc, np.arange(n), np.arange(n), M=n, N=n, K=K)
            err = gemm_ref.err_metric(vals, C_ref, D)
            assert err <= tol(BF16), "moe %s step %d %s err %.3g" % (reading, step, (N, K), err)
            # every covered row was written (no NaN left from the fill)
            assert not t.isnan(C[:int(np.clip(counts, 0, None).sum())]).any().item()


# ---- strided batch (BatchMM)


def batched_case(batch, M, N, K, lda, ldb, ldc, stride_a, stride_b, stride_c, seed):
    """Flat host operands of a strided batch (gaps between matrices stay 0)."""
    A = np.zeros(max((batch - 1) * stride_a + (M - 1) * lda + K, 1) + 8, np.uint16)
    B = np.zeros(max((batch - 1) * stride_b + (K - 1) * ldb + N, 1) + 8, np.uint16)
    for b in range(batch):
        if M and K:
            np.lib.stride_tricks.as_strided(A[b * stride_a:], shape=(M, K), strides=(lda * 2, 2))[...] = \
                gen.uniform_bf16(M, K, seed + 2 * b)
        if K and N and (stride_b or b == 0):
            np.lib.stride_tricks.as_strided(B[b * stride_b:], shape=(K, N), strides=(ldb * 2, 2))[...] = \
                gen.uniform_bf16(K, N, seed + 2 * b + 1)
    return A, B


def run_batched(plan, A, B, batch, M, N, K, lda, ldb, ldc, stride_a, stride_b, stride_c, dtype, addmm=None):
    """One adaptcore_batched_matmul (or, with addmm = (c_old, alpha, beta,
    bias), adaptcore_batched_addmm with C holding c_old: (batch, M, N) fp32
    values or 16-bit patterns); returns (values (batch, M, N), every element
    outside the C matrices still holds its canary)."""
    t = torch()
    n = (batch - 1) * stride_c + (M - 1) * ldc + N + 2 * ldc
    if dtype == F32:
        host = np.full(n, F32_CANARY, np.float32)
    else:
        host = np.full(n, BF16_CANARY, np.uint16)
    if addmm is not None:
        for b in range(batch):
            for i in range(M):
                o = ldc + b * stride_c + i * ldc
                host[o:o + N] = addmm[0][b, i]
    if dtype == F32:
        dev = t.from_numpy(host.copy()).to("cuda")
        addr = dev.data_ptr() + 4 * ldc
    else:
        dev = t.from_numpy(host.view(np.int16).copy()).to("cuda")
        addr = dev.data_ptr() + 2 * ldc
    Ad = t.from_numpy(A.view(np.int16)).to("cuda")
    Bd = t.from_numpy(B.view(np.int16)).to("cuda")
    if addmm is None:
        ac.adaptcore_batched_matmul(plan, Ad.data_ptr(), lda, stride_a, Bd.data_ptr(), ldb, stride_b, addr, ldc,
                                    stride_c, 0)
    else:
        _, alpha, beta, bias = addmm
        bd = t.from_numpy(np.ascontiguousarray(bias, np.float32)).to("cuda") if bias is not None else None
        ac.adaptcore_batched_addmm(plan, Ad.data_ptr(), lda, stride_a, Bd.data_ptr(), ldb, stride_b, addr, ldc,
                                   stride_c, alpha, beta, bd.data_ptr() if bd is not None else 0, 0)
    t.cuda.synchronize()
    raw = dev.cpu().numpy()
    raw = raw if dtype == F32 else raw.view(np.uint16)
    inside = np.zeros(n, bool)
    vals = np.zeros((batch, M, N))
    for b in range(batch):
        for i in range(M):
            o = ldc + b * stride_c + i * ldc
            inside[o:o + N] = True
            row = raw[o:o + N]
            vals[b, i] = row.astype(np.float64) if dtype == F32 else gemm_ref.decode(np.ascontiguousarray(row))
    canary = F32_CANARY if dtype == F32 else BF16_CANARY
    return vals, bool(np.all(raw[~inside] == canary))


def batched_keys(batch, M, N, K, dtype):
    keys = []
    for cfg in range(16):
        for sw in (0, 1):
            key = ac.AC_FAMILY_BATCHED | (cfg << 4) | (sw << 12) | (1 << 16) | (dtype << 48)
            try:
                ac.adaptcore_batched_plan_variant(batch, M, N, K, dtype, 0, key)
            except ac.AdaptCoreError:
                continue
            keys.append(key)
    return keys


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
def test_every_batched_configuration(dtype):
    """Five batches of 70 x 300 x 197 with padded leading dimensions and gaps
    between the matrices (which must keep their canaries)."""
    batch, M, N, K = 5, 70, 300, 197
    lda, ldb, ldc = K + 3, N + 5, N + 7
    sa, sb, sc = M * lda + 11, K * ldb + 13, M * ldc + 17
    A, B = batched_case(batch, M, N, K, lda, ldb, ldc, sa, sb, sc, seed=31)
    C_ref, D = grouped_ref.batched_gemm(A, B, batch, M, N, K, lda, ldb, sa, sb)
    keys = batched_keys(batch, M, N, K, dtype)
    assert len(keys) >= 10
    for key in keys:
        plan = ac.adaptcore_batched_plan_variant(batch, M, N, K, dtype, 0, key)
        note("batched", hex(key), ac.adaptcore_plan_kernels(plan))
        vals, ok = run_batched(plan, A, B, batch, M, N, K, lda, ldb, ldc, sa, sb, sc, dtype)
        assert ok, "write outside the C matrices %s" % hex(key)
        err = gemm_ref.err_metric(vals.reshape(-1, N), C_ref.reshape(-1, N), D.reshape(-1, N))
        assert err <= tol(dtype), "err %.3g %s" % (err, hex(key))


@pytest.mark.parametrize("case", [
    (1, 300, 200, 100, False),     # one batch: a plain product
    (64, 32, 32, 32, False),       # many small matrices
    (12, 17, 5, 3, False),         # N < 8 and K < 8
    (9, 100, 64, 48, True),        # shared B (stride_b = 0)
    (4, 256, 256, 256, False),     # whole tiles
], ids=lambda c: "b%d_%dx%dx%d%s" % (c[0], c[1], c[2], c[3], "_sharedB" if c[4] else ""))
def test_batched_default_plans(case):
    batch, M, N, K, shared = case
    lda, ldb, ldc = K, N, N
    sa, sb, sc = M * K, (0 if shared else K * N), M * N
    A, B = batched_case(batch, M, N, K, lda, ldb, ldc, sa, sb, sc, seed=batch + M)
    C_ref, D = grouped_ref.batched_gemm(A, B, batch, M, N, K, lda, ldb, sa, sb)
    for dtype in (F32, BF16):
        plan = ac.adaptcore_batched_plan(batch, M, N, K, dtype)
        vals, ok = run_batched(plan, A, B, batch, M, N, K, lda, ldb, ldc, sa, sb, sc, dtype)
        assert ok
        err = gemm_ref.err_metric(vals.reshape(-1, N), C_ref.reshape(-1, N), D.reshape(-1, N))
        assert err <= tol(dtype), (case, dtype, err)


@pytest.mark.parametrize("dtype", [F32, BF16], ids=["f32out", "bf16out"])
def test_batched_addmm_every_configuration(dtype):
    """The batched product with the AddMM epilogue (alpha, beta, a bias row
    shared by the batches) on every batched configuration, padded leading
    dimensions and gaps between the matrices; then beta = 0 with NaN in C."""
    batch, M, N, K = 4, 70, 300, 197
    lda, ldb, ldc = K + 3, N + 5, N + 7
    sa, sb, sc = M * lda + 11, K * ldb + 13, M * ldc + 17
    A, B = batched_case(batch, M, N, K, lda, ldb, ldc, sa, sb, sc, seed=41)
    if dtype == F32:
        stored = gen.uniform_f32(batch * M, N, 42, -2.0, 2.0).reshape(batch, M, N)
        old = stored.astype(np.float64)
    else:
        stored = gen.uniform_bf16(batch * M, N, 42, -2.0, 2.0).reshape(batch, M, N)
        old = gemm_ref.decode(stored.reshape(-1, N)).reshape(batch, M, N)
    bias = gen.uniform_f32(1, N, 43).reshape(-1)
    C_ref, D = addmm_ref.batched_addmm(A, B, old, batch, M, N, K, lda, ldb, sa, sb, -0.75, 1.5, bias)
    for key in batched_keys(batch, M, N, K, dtype):
        plan = ac.adaptcore_batched_plan_variant(batch, M, N, K, dtype, 0, key)
        vals, ok = run_batched(plan, A, B, batch, M, N, K, lda, ldb, ldc, sa, sb, sc, dtype,
                               addmm=(stored, -0.75, 1.5, bias))
        assert ok, "write outside the C matrices %s" % hex(key)
        err = gemm_ref.err_metric(vals.reshape(-1, N), C_ref.reshape(-1, N), D.reshape(-1, N))
        assert err <= tol(dtype), "err %.3g %s" % (err, hex(key))
    nan = np.full_like(stored, np.nan) if dtype == F32 else np.full_like(stored, 0x7FC0)
    C_ref, D = addmm_ref.batched_addmm(A, B, None, batch, M, N, K, lda, ldb, sa, sb, 2.0, 0.0, bias)
    plan = ac.adaptcore_batched_plan(batch, M, N, K, dtype)
    vals, ok = run_batched(plan, A, B, batch, M, N, K, lda, ldb, ldc, sa, sb, sc, dtype, addmm=(nan, 2.0, 0.0, bias))
    err = gemm_ref.err_metric(vals.reshape(-1, N), C_ref.reshape(-1, N), D.reshape(-1, N))
    assert ok and err <= tol(dtype), err


def test_batched_k_zero():
    batch, M, N = 3, 20, 24
    A = np.zeros(8, np.uint16)
    B = np.zeros(8, np.uint16)
    plan = ac.adaptcore_batched_plan(batch, M, N, 0, F32)
    vals, ok = run_batched(plan, A, B, batch, M, N, 0, 1, N, N, 0, 0, M * N + 5, F32)
    assert ok and not vals.any()



def test_fp16_grouped_and_batched():
    """The grouped and batched products with fp16 inputs and output."""
    F16 = ac.AC_F16_F16OUT
    counts, rows, N, K = [90, 0, 37, 200, 1], 400, 200, 130
    A = gen.uniform_f16(rows, K, 41)
    mats = [gen.uniform_f16(K, N, 42 + g) for g in range(len(counts))]
    B = np.concatenate([m.reshape(-1) for m in mats])
    t = torch()
    Ad = t.from_numpy(A.view(np.int16)).cuda()
    Bd = t.from_numpy(B.view(np.int16)).cuda()
    cnt = t.from_numpy(np.asarray(counts, np.int32)).cuda()
    Cd = t.zeros(rows * N, dtype=t.int16, device="cuda")
    plan = ac.adaptcore_grouped_plan(rows, len(counts), N, K, F16)
    assert ac.adaptcore_plan_kernels(plan)[0].startswith("f16::k_grouped<")
    ac.adaptcore_grouped_matmul(plan, cnt.data_ptr(), Ad.data_ptr(), K, Bd.data_ptr(), N, K * N, Cd.data_ptr(), N, 0)
    t.cuda.synchronize()
    got = gemm_ref.decode(Cd.cpu().numpy().view(np.uint16).reshape(rows, N), fmt="fp16")
    C_ref, D, cov = grouped_ref.grouped_gemm(A, B, counts, rows, N, K, K, N, K * N, fmt="fp16")
    got = np.where(np.abs(got - C_ref) <= 2.0 ** -25, C_ref, got)
    assert gemm_ref.err_metric(got[cov], C_ref[cov], D[cov]) <= gemm_ref.TOL["fp16"]
    assert not got[~cov].any()
    # batched: contiguous batches of 80 rows
    batch, M = 5, 80
    plan = ac.adaptcore_batched_plan(batch, M, N, K, F16)
    Cd.zero_()
    ac.adaptcore_batched_matmul(plan, Ad.data_ptr(), K, M * K, Bd.data_ptr(), N, K * N, Cd.data_ptr(), N, M * N, 0)
    t.cuda.synchronize()
    got = gemm_ref.decode(Cd.cpu().numpy().view(np.uint16)[:batch * M * N].reshape(batch, M, N), fmt="fp16")
    C_ref, D = grouped_ref.batched_gemm(A, B, batch, M, N, K, K, N, M * K, K * N, fmt="fp16")
    got = np.where(np.abs(got - C_ref) <= 2.0 ** -25, C_ref, got)
    assert gemm_ref.err_metric(got.reshape(-1, N), C_ref.reshape(-1, N), D.reshape(-1, N)) <= gemm_ref.TOL["fp16"]


def test_tensor_bindings():
    """bmm_tensors (plain, with the AddMM epilogue, and with B broadcast over
    the batch) and grouped_mm_tensors (per-group and shared B) against the
    batched and grouped oracles."""
    t = torch()
    batch, M, N, K = 3, 50, 70, 90
    A = gen.uniform_bf16(batch * M, K, 71)
    B = gen.uniform_bf16(batch * K, N, 72)
    Ad = t.from_numpy(A.view(np.int16)).cuda().view(t.bfloat16).view(batch, M, K)
    Bd = t.from_numpy(B.view(np.int16)).cuda().view(t.bfloat16).view(batch, K, N)
    C = t.empty(batch, M, N, dtype=t.float32, device="cuda")
    ac.bmm_tensors(Ad, Bd, C)
    t.cuda.synchronize()
    C_ref, D = grouped_ref.batched_gemm(A.reshape(-1), B.reshape(-1), batch, M, N, K, K, N, M * K, K * N)
    err = gemm_ref.err_metric(C.cpu().numpy().reshape(-1, N).astype(np.float64), C_ref.reshape(-1, N),
                              D.reshape(-1, N))
    assert err <= tol(F32), err
    # AddMM epilogue on the same operands
    old = gen.uniform_f32(batch * M, N, 73).reshape(batch, M, N)
    bias = gen.uniform_f32(1, N, 74).reshape(-1)
    C = t.from_numpy(old.copy()).cuda()
    ac.bmm_tensors(Ad, Bd, C, alpha=0.5, beta=-1.0, bias=t.from_numpy(bias).cuda())
    t.cuda.synchronize()
    R, DR = addmm_ref.batched_addmm(A.reshape(-1), B.reshape(-1), old.astype(np.float64), batch, M, N, K, K, N, M * K,
                                    K * N, 0.5, -1.0, bias)
    err = gemm_ref.err_metric(C.cpu().numpy().reshape(-1, N).astype(np.float64), R.reshape(-1, N), DR.reshape(-1, N))
    assert err <= tol(F32), err
    # B broadcast over the batch (batch stride 0)
    Bb = Bd[0:1].expand(batch, K, N)
    C = t.empty(batch, M, N, dtype=t.float32, device="cuda")
    ac.bmm_tensors(Ad, Bb, C)
    t.cuda.synchronize()
    C_ref, D = grouped_ref.batched_gemm(A.reshape(-1), B.reshape(-1), batch, M, N, K, K, N, M * K, 0)
    err = gemm_ref.err_metric(C.cpu().numpy().reshape(-1, N).astype(np.float64), C_ref.reshape(-1, N),
                              D.reshape(-1, N))
    assert err <= tol(F32), err
    # grouped: 3 groups over 140 rows (the last 10 rows uncovered)
    counts = np.array([60, 0, 70], np.int32)
    rows = 140
    Ag = gen.uniform_bf16(rows, K, 75)
    Agd = t.from_numpy(Ag.view(np.int16)).cuda().view(t.bfloat16)
    cnt = t.from_numpy(counts).cuda()
    for shared in (False, True):
        Bg = Bd[0] if shared else Bd
        Cg = t.zeros(rows, N, dtype=t.float32, device="cuda")
        ac.grouped_mm_tensors(Agd, Bg, cnt, Cg)
        t.cuda.synchronize()
        R, DR, cov = grouped_ref.grouped_gemm(Ag, B.reshape(-1), counts, rows, N, K, K, N, 0 if shared else K * N)
        got = Cg.cpu().numpy().astype(np.float64)
        err = gemm_ref.err_metric(got[cov], R[cov], DR[cov])
        assert err <= tol(F32) and not got[~cov].any(), (shared, err)
