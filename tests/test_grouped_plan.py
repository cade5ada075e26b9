"""Grouped-product planning and C-ABI validation (no GPU).

The grouped kernel's grid must cover every row tile for ANY device count
array (the host never sees the counts): checked here against brute force
over random splits, including negative and over-capacity counts. Plans are
cached, forced configurations round-trip through their keys, and the entry
points reject bad arguments before any GPU work.
"""
import numpy as np
import pytest

import paper_2608_10803_amd as ac

GROUPED_TILES = {(256, 128), (128, 256), (128, 128), (128, 64), (64, 128), (64, 64)}


def _row_tiles(counts, rows, bm):
    """Row tiles of a split under the stated readings (negative -> 0, rows past
    the capacity dropped), written out directly."""
    total, p = 0, 0
    for c in counts:
        c = max(int(c), 0)
        s, e = min(p, rows), min(p + c, rows)
        total += -(-(e - s) // bm)
        p += c
    return total


def test_plan_fields_and_cache():
    h = ac.adaptcore_grouped_plan(8192, 64, 1536, 4096)
    assert h == ac.adaptcore_grouped_plan(8192, 64, 1536, 4096)
    d = ac.adaptcore_plan_info(h)
    assert d["family_name"] == "grouped" and d["groups"] == 64 and d["M"] == 8192
    assert (d["tile_m"], d["tile_n"]) in GROUPED_TILES
    assert d["pn"] == -(-1536 // d["tile_n"]) and d["grid_x"] == d["pm"] * d["pn"] and d["pk"] == 1
    assert d["workspace_bytes"] == 0 and d["predicted_s"] > 0
    names = ac.adaptcore_plan_kernels(h)
    assert len(names) == 1 and names[0].startswith("k_grouped<%d, %d, " % (d["tile_m"], d["tile_n"]))
    # a plain plan of the same dimensions is a different object
    assert ac.adaptcore_plan(8192, 1536, 4096) != h


@pytest.mark.parametrize("seed", range(4))
def test_grid_covers_every_split(seed):
    rng = np.random.default_rng(seed)
    for _ in range(60):
        G = int(rng.integers(1, 300))
        rows = int(rng.integers(1, 5000))
        N, K = int(rng.integers(1, 5000)), int(rng.integers(0, 5000))
        d = ac.adaptcore_plan_info(ac.adaptcore_grouped_plan(rows, G, N, K))
        bm = d["tile_m"]
        splits = [rng.multinomial(rows, np.ones(G) / G), rng.integers(-3, 2 * rows // G + 3, G),
                  np.r_[np.zeros(G - 1, int), rows], np.ones(G, int) * (rows // G + 1)]
        w = rng.zipf(1.2, G).astype(float)
        splits.append(rng.multinomial(rows, w / w.sum()))
        for counts in splits:
            assert _row_tiles(counts, rows, bm) <= d["pm"], (rows, G, bm, d["pm"])
        # the bound is reached by one row in each of min(G, rows) groups plus the rest in one group
        ne = min(G, rows)
        worst = np.r_[np.ones(ne - 1, int), rows - ne + 1, np.zeros(G - ne, int)]
        assert _row_tiles(worst, rows, bm) <= d["pm"]


def test_forced_configurations_round_trip():
    for cfg in range(16):
        for sw in (0, 1):
            key = ac.AC_FAMILY_GROUPED | (cfg << 4) | (sw << 12) | (1 << 16) | (ac.AC_BF16_BF16OUT << 48)
            try:
                h = ac.adaptcore_grouped_plan_variant(700, 9, 300, 197, ac.AC_BF16_BF16OUT, 0, key)
            except ac.AdaptCoreError:
                continue
            d = ac.adaptcore_plan_info(h)
            assert d["variant_key"] == key and d["swizzle"] == sw
            assert (d["tile_m"], d["tile_n"]) in GROUPED_TILES
    # a plain-family key is not a grouped configuration
    with pytest.raises(ac.AdaptCoreError):
        ac.adaptcore_grouped_plan_variant(700, 9, 300, 197, ac.AC_BF16_BF16OUT, 0,
                                          (3 << 4) | (1 << 16) | (ac.AC_BF16_BF16OUT << 48))


def test_argument_validation():
    with pytest.raises(ac.AdaptCoreError):
        ac.adaptcore_grouped_plan(10, -1, 4, 4)
    with pytest.raises(ac.AdaptCoreError):
        ac.adaptcore_grouped_plan(10, (1 << 20) + 1, 4, 4)
    with pytest.raises(ac.AdaptCoreError):
        ac.adaptcore_grouped_plan(-1, 3, 4, 4)
    with pytest.raises(ac.AdaptCoreError) as e:
        ac.adaptcore_grouped_plan(10, 3, 4, 4, 9)
    assert e.value.status == ac.AC_ERR_UNSUPPORTED
    hg = ac.adaptcore_grouped_plan(64, 4, 32, 16)
    hp = ac.adaptcore_plan(64, 32, 16)
    # the two kinds of plan are not interchangeable
    with pytest.raises(ac.AdaptCoreError) as e:
        ac.adaptcore_matmul(hg, 0x1000, 16, 0x2000, 32, 0x3000, 32)
    assert e.value.status == ac.AC_ERR_INVALID_VALUE
    with pytest.raises(ac.AdaptCoreError) as e:
        ac.adaptcore_grouped_matmul(hp, 0x4000, 0x1000, 16, 0x2000, 32, 512, 0x3000, 32)
    assert e.value.status == ac.AC_ERR_INVALID_VALUE
    good = (0x4000, 0x1000, 16, 0x2000, 32, 512, 0x3000, 32)
    bad = [
        (0x4000, 0x1000, 15, 0x2000, 32, 512, 0x3000, 32),   # lda < K
        (0x4000, 0x1000, 16, 0x2000, 31, 512, 0x3000, 32),   # ldb < N
        (0x4000, 0x1000, 16, 0x2000, 32, 512, 0x3000, 31),   # ldc < N
        (0x4000, 0x1000, 16, 0x2000, 32, -1, 0x3000, 32),    # stride_b < 0
        (0x4000, 0x1000, 16, 0x2000, 32, 1 << 40, 0x3000, 32),
        (0, 0x1000, 16, 0x2000, 32, 512, 0x3000, 32),        # null counts
        (0x4002, 0x1000, 16, 0x2000, 32, 512, 0x3000, 32),   # misaligned counts
        (0x4000, 0x1001, 16, 0x2000, 32, 512, 0x3000, 32),   # misaligned A
        (0x4000, 0x1000, 16, 0x2000, 32, 512, 0, 32),        # null C
    ]
    for args in bad:
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_grouped_matmul(hg, *args)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE, args
    # the AddMM form: the same checks, plus finite scalars, an aligned bias and its stride
    for extra in [(float("nan"), 1.0, 0, 0), (1.0, 1.0, 0x5002, 0), (1.0, 1.0, 0x5000, -1), (1.0, 1.0, 0x5000, 1 << 40)]:
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_grouped_addmm(hg, *good, *extra)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE, extra
    for args in bad:
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_grouped_addmm(hg, *args, 1.0, 0.0, 0, 0)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE, args
    for args in [(0x4000, 0x1000, 1 << 23, 0x2000, 32, 512, 0x3000, 32),
                 (0x4000, 0x1000, 16, 0x2000, 1 << 23, 512, 0x3000, 32)]:
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_grouped_matmul(hg, *args)
        assert e.value.status == ac.AC_ERR_UNSUPPORTED
    # nothing to compute: no launch, success anywhere
    for h in [ac.adaptcore_grouped_plan(0, 4, 32, 16), ac.adaptcore_grouped_plan(64, 0, 32, 16),
              ac.adaptcore_grouped_plan(64, 4, 0, 16)]:
        ac.adaptcore_grouped_matmul(h, *good)
    assert good  # the good tuple is only launched on a GPU (tests/test_gpu_grouped.py)


# ---- strided batch (BatchMM) on the grouped kernel


def test_batched_plan_fields_and_cache():
    h = ac.adaptcore_batched_plan(64, 130, 300, 197)
    assert h == ac.adaptcore_batched_plan(64, 130, 300, 197)
    d = ac.adaptcore_plan_info(h)
    assert d["family_name"] == "batched" and d["groups"] == 64 and (d["M"], d["N"], d["K"]) == (130, 300, 197)
    tpg = -(-130 // d["tile_m"])
    assert d["pm"] == 64 * tpg and d["pn"] == -(-300 // d["tile_n"]) and d["grid_x"] == d["pm"] * d["pn"]
    assert ac.adaptcore_plan_kernels(h)[0].startswith("k_grouped<")
    # distinct from the grouped plan of the same numbers
    assert h != ac.adaptcore_grouped_plan(130, 64, 300, 197)
    for cfg in range(16):
        key = ac.AC_FAMILY_BATCHED | (cfg << 4) | (1 << 12) | (1 << 16) | (ac.AC_BF16_BF16OUT << 48)
        try:
            hv = ac.adaptcore_batched_plan_variant(64, 130, 300, 197, ac.AC_BF16_BF16OUT, 0, key)
        except ac.AdaptCoreError:
            continue
        assert ac.adaptcore_plan_info(hv)["variant_key"] == key


def test_batched_argument_validation():
    with pytest.raises(ac.AdaptCoreError):
        ac.adaptcore_batched_plan(-1, 4, 4, 4)
    with pytest.raises(ac.AdaptCoreError):
        ac.adaptcore_batched_plan((1 << 24) + 1, 4, 4, 4)
    hb = ac.adaptcore_batched_plan(3, 16, 32, 8)
    hg = ac.adaptcore_grouped_plan(48, 3, 32, 8)
    hp = ac.adaptcore_plan(16, 32, 8)
    ok = (0x1000, 8, 128, 0x2000, 32, 256, 0x3000, 32, 512)
    # every kind of plan only runs through its own entry point
    for h in (hg, hp):
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_batched_matmul(h, *ok)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE
    for f, args in [(ac.adaptcore_matmul, (0x1000, 8, 0x2000, 32, 0x3000, 32)),
                    (ac.adaptcore_grouped_matmul, (0x4000, 0x1000, 8, 0x2000, 32, 256, 0x3000, 32))]:
        with pytest.raises(ac.AdaptCoreError) as e:
            f(hb, *args)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE
    bad = [
        (0x1000, 7, 128, 0x2000, 32, 256, 0x3000, 32, 512),     # lda < K
        (0x1000, 8, -1, 0x2000, 32, 256, 0x3000, 32, 512),      # negative stride
        (0x1000, 8, 128, 0x2000, 32, 256, 0x3000, 32, 1 << 40),
        (0x1000, 8, 128, 0x2000, 32, 256, 0x3000, 32, 15 * 32 + 31),  # C matrices overlap
        (0x1000, 8, 128, 0x2000, 32, 256, 0x3001, 32, 512),     # misaligned C (bf16: 2 bytes)
        (0x1000, 8, 128, 0x2000, 32, 256, 0, 32, 512),          # null C
    ]
    for args in bad:
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_batched_matmul(hb, *args)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE, args
    with pytest.raises(ac.AdaptCoreError) as e:
        ac.adaptcore_batched_matmul(hb, 0x1000, 1 << 23, 128, 0x2000, 32, 256, 0x3000, 32, 512)
    assert e.value.status == ac.AC_ERR_UNSUPPORTED
    # the AddMM form: the same checks, plus finite scalars and an aligned bias
    for alpha, beta, bias in [(float("nan"), 1.0, 0), (1.0, float("-inf"), 0), (1.0, 1.0, 0x5001)]:
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_batched_addmm(hb, *ok, alpha, beta, bias)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE
    for args in bad:
        with pytest.raises(ac.AdaptCoreError) as e:
            ac.adaptcore_batched_addmm(hb, *args, 1.0, 0.0, 0)
        assert e.value.status == ac.AC_ERR_INVALID_VALUE, args
    # the smallest stride that keeps the C matrices apart is accepted before any GPU work is needed
    for h in (ac.adaptcore_batched_plan(0, 16, 32, 8), ac.adaptcore_batched_plan(3, 0, 32, 8)):
        ac.adaptcore_batched_matmul(h, 0x1000, 8, 128, 0x2000, 32, 256, 0x3000, 32, 15 * 32 + 32)
