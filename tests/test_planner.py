"""Planner, plan cache and C-ABI checks that need no GPU.

The planner's taxonomy and latency-model closed forms are compared with the
oracle (oracle/taxonomy.py), which is itself pinned to the paper's worked
cases and to brute force. The cache is checked for identity of plans, O(1)
lookup cost and thread safety; the ABI for argument validation and for
exporting every declared symbol.
"""
import ctypes
import os
import random
import re
import threading

import pytest

import paper_2608_10803_amd as ac
from oracle import taxonomy as tx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    hdr = open(os.path.join(ROOT, "include", "adaptcore.h")).read()
    names = set(re.findall(r"\b(adaptcore_[a-z_]+)\s*\(", hdr))
    assert len(names) >= 15
    L = ctypes.CDLL(ac._lib.LIB_PATH)
    missing = [n for n in sorted(names) if not hasattr(L, n)]
    assert not missing, missing
    # and the binding exposes the same names
    assert all(hasattr(ac, n) for n in names)


@pytest.mark.parametrize("case", [
    (1024, 1024, 1024, 128, 256, 1024, 128, 256, 64),
    (4096, 4096, 1024, 256, 256, 1024, 256, 256, 64),
    (128, 128, 4096, 64, 64, 1024, 64, 64, 64),
    (256, 256, 8192, 256, 256, 2048, 256, 256, 64),
])
def test_paper_cases_through_abi(case):
    """Section 4.3 cases on 16 cores / 128 KB, through the library."""
    M, N, K, m, n, k, m1, n1, k1 = case
    got = ac.adaptcore_taxonomy(M, N, K, m, n, k, m1, n1, k1, 16, 128 * 1024)
    assert got["cls"] == tx.classify(M, N, m, n, m1, n1, 16, 128 * 1024)
    assert got["acc_bytes"] == tx.acc_tile_bytes(m1, n1)


def test_taxonomy_parity_random():
    rnd = random.Random(5)
    for _ in range(3000):
        M, N, K = (rnd.randint(1, 5000) for _ in range(3))
        m, n = rnd.choice([16, 32, 64, 128, 256]), rnd.choice([16, 32, 64, 128, 256])
        k = rnd.randint(1, K)
        m1, n1 = rnd.choice([16, 32, 64, 128, 256, 512]), rnd.choice([16, 32, 64, 128, 256])
        k1 = rnd.randint(1, 256)
        n_core = rnd.choice([16, 24, 256])
        s_acc = rnd.choice([128 * 1024, 256 * 1024])
        got = ac.adaptcore_taxonomy(M, N, K, m, n, k, m1, n1, k1, n_core, s_acc)
        pm, pn, pk = tx.task_counts(M, N, K, m, n, k)
        assert (got["pm"], got["pn"], got["pk"]) == (pm, pn, pk)
        cls = tx.classify(M, N, m, n, m1, n1, n_core, s_acc)
        assert got["cls"] == cls
        assert got["read_bytes"] == pytest.approx(float(tx.read_volume(M, N, K, m1, n1)), rel=1e-12)
        assert got["write_bytes"] == float(tx.write_volume(cls, M, N, K, k, k1))


def test_schedule_parity():
    rnd = random.Random(6)
    for _ in range(2000):
        Q, L = rnd.randint(1, 8), rnd.randint(1, 64)
        tm, tp, td = (rnd.randint(0, 1000) / 8 for _ in range(3))
        assert ac.adaptcore_schedule(0, Q, L, tm, tp, td) == float(tx.t_baseline(L, tm, tp, td))
        assert ac.adaptcore_schedule(1, Q, L, tm, tp, td) == float(tx.t_double_buffer(L, tm, tp, td))
        assert ac.adaptcore_schedule(2, Q, L, tm, tp, td) == float(tx.t_preload(Q, L, tm, tp, td))


def test_shape_classes_follow_the_taxonomy():
    # spatially saturated shapes are Common, starved ones MultiCoreSplitK
    p = ac.adaptcore_plan_info(ac.adaptcore_plan(8192, 8192, 1024))
    assert p["cls_name"] == "Common" and p["pk"] == 1
    p = ac.adaptcore_plan_info(ac.adaptcore_plan(128, 128, 65536))
    assert p["cls_name"] == "MultiCoreSplitK" and p["pk"] > 1
    # a K that cannot be split falls back to the Common kernel inside the template
    p = ac.adaptcore_plan_info(ac.adaptcore_plan(100, 100, 5))
    assert p["pk"] == 1


def test_plan_cache_identity_and_stats():
    ac.adaptcore_cache_clear()
    s0 = ac.adaptcore_stats()
    h1 = ac.adaptcore_plan(777, 333, 999, ac.AC_BF16_F32OUT)
    h2 = ac.adaptcore_plan(777, 333, 999, ac.AC_BF16_F32OUT)
    h3 = ac.adaptcore_plan(777, 333, 999, ac.AC_BF16_BF16OUT)
    assert h1 == h2 and h1 != h3
    s1 = ac.adaptcore_stats()
    assert s1["misses"] - s0["misses"] == 2 and s1["hits"] - s0["hits"] == 1
    d = ac.adaptcore_plan_info(h1)
    assert (d["M"], d["N"], d["K"], d["dtype"]) == (777, 333, 999, 0)
    # large dimensions go through the exact fallback map
    hb = ac.adaptcore_plan(1, 1 << 20, 3)
    assert hb == ac.adaptcore_plan(1, 1 << 20, 3)
    assert ac.adaptcore_plan_info(hb)["N"] == 1 << 20


def test_lookup_is_constant_time_and_fast():
    t_small = ac.adaptcore_bench_lookup(10, 200000)
    t_big = ac.adaptcore_bench_lookup(20000, 200000)
    assert t_small < 1000 and t_big < 1000  # < 1 us per cached lookup
    assert t_big < 20 * max(t_small, 10.0)


def test_concurrent_planning_returns_one_plan_per_shape():
    ac.adaptcore_cache_clear()
    shapes = [(m, n, k) for m in (3, 50, 700) for n in (9, 300) for k in (17, 4096)]
    res = {}
    lock = threading.Lock()

    def worker(seed):
        rnd = random.Random(seed)
        for _ in range(200):
            s = rnd.choice(shapes)
            h = ac.adaptcore_plan(*s)
            with lock:
                res.setdefault(s, set()).add(h)

    ts = [threading.Thread(target=worker, args=(i,)) for i in range(8)]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert all(len(v) == 1 for v in res.values())


def test_argument_validation():
    with pytest.raises(ac.AdaptCoreError):
        ac.adaptcore_plan(-1, 4, 4)
    with pytest.raises(ac.AdaptCoreError) as e:
        ac.adaptcore_plan(4, 4, 4, 7)
    assert e.value.status == ac.AC_ERR_UNSUPPORTED
    with pytest.raises(ac.AdaptCoreError):
        ac.adaptcore_plan(4, 4, 4, ac.AC_BF16_F32OUT, 4)
    h = ac.adaptcore_plan(64, 32, 16)
    # leading dimensions shorter than the rows are rejected before any GPU work
    for args in [(0x1000, 15, 0x2000, 32, 0x3000, 32), (0x1000, 16, 0x2000, 31, 0x3000, 32),
                 (0x1000, 16, 0x2000, 32, 0x3000, 31), (0x1001, 16, 0x2000, 32, 0x3000, 32),
                 (0, 16, 0x2000, 32, 0x3000, 32)]:
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_matmul(h, *args)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE
    # leading dimensions at or past 2^23 are unsupported (32-bit tile offsets)
    for args in [(0x1000, 1 << 23, 0x2000, 32, 0x3000, 32), (0x1000, 16, 0x2000, 1 << 23, 0x3000, 32)]:
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_matmul(h, *args)
        assert e.value.status == ac.AC_ERR_UNSUPPORTED
    # an empty output launches nothing and succeeds anywhere
    ac.adaptcore_matmul(ac.adaptcore_plan(0, 5, 7), 0, 7, 0x2000, 5, 0x3000, 5)
    with pytest.raises(ac.AdaptCoreError):
        ac.adaptcore_matmul(0, 0x1000, 16, 0x2000, 32, 0x3000, 32)


def test_addmm_argument_validation():
    h = ac.adaptcore_plan(64, 32, 16)
    good = (0x1000, 16, 0x2000, 32, 0x3000, 32)
    # non-finite scalars and a misaligned bias are rejected before any GPU work
    for alpha, beta, bias in [(float("nan"), 1.0, 0), (1.0, float("inf"), 0), (1.0, 1.0, 0x4002)]:
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_addmm(h, *good, alpha, beta, bias)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE
    # the plain product's checks apply unchanged
    with pytest.raises(ac.AdaptCoreError) as e:
        ac.adaptcore_addmm(h, 0x1000, 15, 0x2000, 32, 0x3000, 32, 1.0, 1.0, 0)
    assert e.value.status == ac.AC_ERR_INVALID_VALUE
    with pytest.raises(ac.AdaptCoreError) as e:
        ac.adaptcore_addmm(h, 0x1000, 1 << 23, 0x2000, 32, 0x3000, 32, 1.0, 1.0, 0)
    assert e.value.status == ac.AC_ERR_UNSUPPORTED
    # grouped and batched plans only run through their own entry points
    for hp in (ac.adaptcore_grouped_plan(64, 4, 32, 16), ac.adaptcore_batched_plan(4, 16, 32, 16)):
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_addmm(hp, *good, 1.0, 0.0, 0)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE
    # an empty output launches nothing and succeeds anywhere
    ac.adaptcore_addmm(ac.adaptcore_plan(0, 5, 7), 0, 7, 0x2000, 5, 0x3000, 5, 2.0, 0.5, 0x4000)


def _copies(fam, M, N, K, layouts):
    """The prologue copies a plan of this family makes: (kernel, rows,
    columns) each, in launch order (A first)."""
    a_col, b_col = layouts & 1, layouts & 2
    out = []
    if fam == ac.AC_FAMILY_TALL:  # B read as B^T (N x K): transposed from row-major, copied from column-major
        return [("k_pad16" if b_col else "k_transpose16", N, K)]
    dl = fam == ac.AC_FAMILY_DL
    if a_col:
        out.append(("k_transpose16", M, K))
    elif dl and K % 8:
        out.append(("k_pad16", M, K))
    if b_col and fam != ac.AC_FAMILY_SKINNY_M:
        out.append(("k_transpose16", K, N))
    elif not b_col and dl and N % 8:
        out.append(("k_pad16", K, N))
    return out


def test_layout_plans():
    """Column-major operands: a prologue copy per operand in the workspace
    (after the partials, 256-byte aligned, rows padded to 8), priced in the
    prediction -- except a column-major B under the small-M kernel, which
    reads it in place; the direct-to-LDS kernels also pad unaligned
    row-major operands, and the tall-skinny kernel always reads B's
    transposed copy. Every forced configuration keeps the row-major
    configuration's main kernels after the copies."""
    for (M, N, K) in [(2100, 3000, 200), (640, 1000, 4096), (4, 4096, 4096), (37, 91, 333), (3000, 9, 1000)]:
        for layouts in (1, 2, 3):
            for c in ac.adaptcore_candidates(M, N, K, ac.AC_BF16_BF16OUT, layouts):
                key = c["variant_key"]
                assert (key >> 52) & 3 == layouts
                h = ac.adaptcore_plan_variant(M, N, K, ac.AC_BF16_BF16OUT, layouts, key)
                h0 = ac.adaptcore_plan_variant(M, N, K, ac.AC_BF16_BF16OUT, 0, key & ~(3 << 52))
                d, d0 = ac.adaptcore_plan_info(h), ac.adaptcore_plan_info(h0)
                assert d["layouts"] == layouts
                fam = d["family"]
                skinny = fam == ac.AC_FAMILY_SKINNY_M
                # the split-K partials (stream-K: its fp32 tile slots, as in the row-major plan)
                ws = d["pk"] * M * (-(-N // 8) * 8) * 4 if d["pk"] > 1 else 0
                if fam == ac.AC_FAMILY_STREAMK:
                    ws = d0["workspace_bytes"]
                copies = _copies(fam, M, N, K, layouts)
                for _, rows, cols in copies:
                    ws = -(-ws // 256) * 256 + rows * (-(-cols // 8) * 8) * 2
                assert d["workspace_bytes"] == ws, (layouts, c)
                n0 = len(_copies(fam, M, N, K, 0))
                assert (d["predicted_s"] > d0["predicted_s"]) == (len(copies) > n0) or fam == ac.AC_FAMILY_TALL
                names = ac.adaptcore_plan_kernels(h)
                assert names[:len(copies)] == [k for k, _, _ in copies], (names, copies)
                rest = ac.adaptcore_plan_kernels(h0)[n0:]
                if layouts & 2 and skinny:
                    rest = [n.replace("k_skinny_m<", "k_skinny_m_bt<") for n in rest]
                assert names[len(copies):] == rest, (names, rest)
        # the decode shape with B column-major picks the in-place small-M kernel
        if (M, N, K) == (4, 4096, 4096):
            names = ac.adaptcore_plan_kernels(ac.adaptcore_plan(M, N, K, ac.AC_BF16_BF16OUT, 2))
            assert names[0].startswith("k_skinny_m_bt<"), names
    # K == 0: nothing to copy
    d = ac.adaptcore_plan_info(ac.adaptcore_plan(30, 40, 0, ac.AC_BF16_F32OUT, 3))
    assert d["workspace_bytes"] == 0
    # leading dimensions follow the stored orientation
    h = ac.adaptcore_plan(64, 32, 16, ac.AC_BF16_BF16OUT, 3)
    for args in [(0x1000, 63, 0x2000, 16, 0x3000, 32), (0x1000, 64, 0x2000, 15, 0x3000, 32)]:
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_matmul(h, *args)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE
    # the row pitch of a copy must stay below 2^23 like any operand's
    big = ac.adaptcore_plan(2, 2, (1 << 23) - 3, ac.AC_BF16_F32OUT, 1)
    with pytest.raises(ac.AdaptCoreError) as e:
        ac.adaptcore_matmul(big, 0x1000, 2, 0x2000, 2, 0x3000, 2)
    assert e.value.status == ac.AC_ERR_UNSUPPORTED
    # unknown bits, and grouped and batched products, are refused
    with pytest.raises(ac.AdaptCoreError) as e:
        ac.adaptcore_plan(4, 4, 4, ac.AC_BF16_F32OUT, 4)
    assert e.value.status == ac.AC_ERR_UNSUPPORTED
    for f, args in [(ac.adaptcore_grouped_plan, (64, 4, 32, 16)), (ac.adaptcore_batched_plan, (4, 16, 32, 16))]:
        with pytest.raises(ac.AdaptCoreError) as e:
            f(*args, ac.AC_BF16_F32OUT, 1)
        assert e.value.status == ac.AC_ERR_UNSUPPORTED


def test_candidates_are_legal_and_keys_round_trip():
    hw = ac.adaptcore_get_hw()
    for s in [(1, 4096, 4096), (17, 300, 65536), (512, 512, 512), (3000, 5, 700), (64, 64, 65536),
              (100000, 8, 5), (4096, 4096, 4096), (1, 1, 1)]:
        cands = ac.adaptcore_candidates(*s)
        assert cands, s
        preds = [c["predicted_s"] for c in cands]
        assert preds == sorted(preds)
        best = ac.adaptcore_plan_info(ac.adaptcore_plan(*s))
        assert best["variant_key"] == cands[0]["variant_key"]
        for c in cands[:40]:
            h = ac.adaptcore_plan_variant(*s, ac.AC_BF16_BF16OUT, 0, c["variant_key"])
            d = ac.adaptcore_plan_info(h)
            assert d["variant_key"] == c["variant_key"]
            assert d["predicted_s"] == pytest.approx(c["predicted_s"])
            assert d["workspace_bytes"] <= (2 << 30) + (1 << 20)
            assert d["grid_y"] <= 65535 and d["grid_x"] >= 1
            assert d["pk"] >= 1
    # the small-N kernel walks any K in LDS-sized chunks: no split is forced
    assert any(c["family_name"] == "skinny_n" and c["pk"] == 1 for c in ac.adaptcore_candidates(3000, 5, 70000))
    with pytest.raises(ac.AdaptCoreError):
        ac.adaptcore_plan_variant(5, 5, 5, ac.AC_BF16_BF16OUT, 0, 0xFFFF)
    ac.adaptcore_set_hw(hw)


def test_open_search_is_a_superset():
    hw = ac.adaptcore_get_hw()
    s = (200, 3000, 9000)
    closed = {c["variant_key"] for c in ac.adaptcore_candidates(*s)}
    h2 = ac.adaptcore_get_hw()
    h2.search_open = 1
    h2.enable_streamk = 1
    ac.adaptcore_set_hw(h2)
    try:
        opened = {c["variant_key"] for c in ac.adaptcore_candidates(*s)}
    finally:
        ac.adaptcore_set_hw(hw)
    assert closed < opened


def test_profile_validation_and_cu_count_effect():
    hw = ac.adaptcore_get_hw()
    bad = ac.adaptcore_get_hw()
    bad.n_cu = 0
    with pytest.raises(ac.AdaptCoreError):
        ac.adaptcore_set_hw(bad)
    small = ac.adaptcore_get_hw()
    small.n_cu = 16
    ac.adaptcore_set_hw(small)
    try:
        # with 16 cores, 1024^3 saturates the device (Section 4.3, case 1 analogue)
        assert ac.adaptcore_plan_info(ac.adaptcore_plan(1024, 1024, 1024))["cls_name"] == "Common"
    finally:
        ac.adaptcore_set_hw(hw)
    assert ac.adaptcore_get_hw().n_cu == hw.n_cu


def test_fp16_plans():
    """fp16 inputs plan like bf16 (same model, same configurations), under a
    different key, with the kernels of the fp16 build."""
    for s in [(512, 512, 512), (3, 4096, 4096), (20000, 30000, 100), (7, 5, 3)]:
        for dt16, dtb in [(ac.AC_F16_F32OUT, ac.AC_BF16_F32OUT), (ac.AC_F16_F16OUT, ac.AC_BF16_BF16OUT)]:
            h16, hb = ac.adaptcore_plan(*s, dt16), ac.adaptcore_plan(*s, dtb)
            d16, db = ac.adaptcore_plan_info(h16), ac.adaptcore_plan_info(hb)
            assert h16 != hb and d16["shape_key"] != db["shape_key"]
            assert (d16["family"], d16["tile_m"], d16["tile_n"], d16["pk"]) == (db["family"], db["tile_m"], db["tile_n"], db["pk"])
            k16, kb = ac.adaptcore_plan_kernels(h16), ac.adaptcore_plan_kernels(hb)
            # the prologue copies move 16-bit patterns: shared by both formats
            shared = ("k_pad16", "k_transpose16")
            assert k16 == [k if k in shared else "f16::" + k for k in kb], (k16, kb)
    with pytest.raises(ac.AdaptCoreError) as e:
        ac.adaptcore_plan(4, 4, 4, 4)
    assert e.value.status == ac.AC_ERR_UNSUPPORTED


def test_set_override_is_thread_local_and_leaves_the_cache():
    """adaptcore_set_override forces the configuration of the calling
    thread's adaptcore_plan calls (the exhaustive-search hook, Section 6.6):
    each legal key of a shape comes back through adaptcore_plan, other
    threads still get the model's choice, the shape cache gains no entry and
    its plan is unchanged, an illegal key gives NULL, and 0 restores."""
    s = (700, 900, 3000)
    chosen = ac.adaptcore_plan(*s)
    chosen_key = ac.adaptcore_plan_info(chosen)["variant_key"]
    cands = ac.adaptcore_candidates(*s)
    others = [c["variant_key"] for c in cands if c["variant_key"] != chosen_key][:6]
    assert others
    entries = ac.adaptcore_stats()["entries"]
    seen_other_thread = []
    try:
        for k in others:
            ac.adaptcore_set_override(k)
            assert ac.adaptcore_get_override() == k
            h = ac.adaptcore_plan(*s)
            assert ac.adaptcore_plan_info(h)["variant_key"] == k
            assert h == ac.adaptcore_plan_variant(*s, ac.AC_BF16_BF16OUT, 0, k)
            t = threading.Thread(target=lambda: seen_other_thread.append(
                (ac.adaptcore_get_override(), ac.adaptcore_plan(*s))))
            t.start()
            t.join()
        # a key of another dtype is not legal for a bf16-output shape
        ac.adaptcore_set_override(others[0] & ~(0xF << 48) | (ac.AC_BF16_F32OUT << 48))
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_plan(*s)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE
    finally:
        ac.adaptcore_set_override(0)
    assert ac.adaptcore_get_override() == 0
    assert all(o == 0 and h == chosen for o, h in seen_other_thread)
    assert ac.adaptcore_plan(*s) == chosen
    assert ac.adaptcore_stats()["entries"] == entries


def _with_hw(**fields):
    hw = ac.adaptcore_get_hw()
    h = ac.adaptcore_get_hw()
    for k, v in fields.items():
        setattr(h, k, v)
    ac.adaptcore_set_hw(h)
    return hw


def test_offchip_templates_and_their_candidates():
    """Off-chip accumulation (SingleCoreSplitK / HybridSplitK): with the
    default capacities no menu tile overflows the registers, so the class
    search never offers it (the open search does); with a smaller
    accumulator capacity the templates arise, SingleCoreSplitK keeps k = K
    per workgroup (one workgroup along K) and HybridSplitK also splits K
    across workgroups. Write volume (Eqs. 3 and 5): P_k fp32 partial slices of
    M x N in the workspace, then one output write by the reduction."""
    BF = ac.AC_BF16_BF16OUT
    s = (8192, 8192, 2048)
    assert not [c for c in ac.adaptcore_candidates(*s, BF, 0) if c["family_name"] == "offchip"]
    hw = _with_hw(search_open=1)
    try:
        assert [c for c in ac.adaptcore_candidates(*s, BF, 0) if c["family_name"] == "offchip"]
    finally:
        ac.adaptcore_set_hw(hw)
    hw = _with_hw(s_acc_bytes=128 * 1024)
    try:
        plan = ac.adaptcore_plan_info(ac.adaptcore_plan_variant(*s, BF, 0, ac.adaptcore_candidates(*s, BF, 0)[0]
                                                                ["variant_key"]))
        assert plan["cls_name"] == "SingleCoreSplitK"
        off = [c for c in ac.adaptcore_candidates(*s, BF, 0) if c["family_name"] == "offchip"]
        assert off and all(c["grid_y"] == 1 and c["pk"] >= 2 for c in off)
        for c in off:
            d = ac.adaptcore_plan_info(ac.adaptcore_plan_variant(*s, BF, 0, c["variant_key"]))
            assert d["workspace_bytes"] == d["pk"] * s[0] * s[1] * 4
            assert d["grid_x"] == (-(-s[0] // 256) + 1) // 2 * -(-s[1] // 256)
    finally:
        ac.adaptcore_set_hw(hw)
    hw = _with_hw(s_acc_bytes=32 * 1024)
    try:
        s = (512, 512, 65536)
        cands = ac.adaptcore_candidates(*s, BF, 0)
        assert cands[0]["cls"] == 3  # HybridSplitK
        off = [c for c in cands if c["family_name"] == "offchip"]
        assert any(c["grid_y"] > 1 for c in off) and all(c["pk"] % c["grid_y"] == 0 for c in off)
    finally:
        ac.adaptcore_set_hw(hw)


def test_persistent_256_tile_only_in_the_open_search():
    """The persistent 256 x 256 tile is measured rarely fastest and is left
    out of the class-fixed search; the open search and forced keys keep it."""
    BF = ac.AC_BF16_BF16OUT
    s = (20000, 20000, 128)
    def pp256(cands):
        return [c for c in cands if c["family_name"] == "persist" and c["tile_m"] == 256 and c["tile_n"] == 256]
    assert not pp256(ac.adaptcore_candidates(*s, BF, 0))
    assert [c for c in ac.adaptcore_candidates(*s, BF, 0) if c["family_name"] == "persist"]
    hw = _with_hw(search_open=1)
    try:
        opened = pp256(ac.adaptcore_candidates(*s, BF, 0))
        assert opened
        key = opened[0]["variant_key"]
    finally:
        ac.adaptcore_set_hw(hw)
    assert ac.adaptcore_plan_kernels(ac.adaptcore_plan_variant(*s, BF, 0, key))[0].startswith("k_tile_pp<256, 256")
