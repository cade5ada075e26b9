"""Host checks of the calibration's bookkeeping: the held-out split, the
near-best record filter and the ranking metrics (top-1, regret) that the
design notes quote. The model's predictions come from the planner on the
host; the "measured" times are set here, so every expected figure is known."""
import math

import pytest

import paper_2608_10803_amd as ac
from paper_2608_10803_amd import calibrate as cal

BF16 = ac.AC_BF16_BF16OUT
SHAPES = [(512, 512, 512), (64, 4096, 4096), (3000, 5000, 40)]


def records(times_of):
    """One record per candidate of each shape, with t = times_of(candidate)."""
    out = []
    for M, N, K in SHAPES:
        for c in ac.adaptcore_candidates(M, N, K, BF16, 0):
            out.append(dict(M=M, N=N, K=K, dtype=BF16, key=c["variant_key"], family=c["family_name"],
                            tile_m=c["tile_m"], tile_n=c["tile_n"], pk=c["pk"], grid=c["grid_x"] * c["grid_y"],
                            pred=c["predicted_s"], t=times_of(c)))
    return out


def test_split_is_a_partition():
    keys = {(m, 7, 9, BF16) for m in range(1, 41)}
    train, test = cal.split_shapes(keys)
    assert train | test == keys and not train & test
    assert abs(len(train) - len(test)) <= 1
    assert cal.split_shapes(keys) == (train, test)  # seeded


def test_near_filter_keeps_the_competitive_records():
    recs = [dict(M=1, N=1, K=1, dtype=BF16, t=t) for t in (1.0, 1.2, 1.31, 3.0)]
    recs += [dict(M=2, N=1, K=1, dtype=BF16, t=t) for t in (5.0, 6.4, 6.6)]
    kept = cal.near_records(recs, 1.3)
    assert sorted((r["M"], r["t"]) for r in kept) == [(1, 1.0), (1, 1.2), (2, 5.0), (2, 6.4)]


def test_perfect_model_ranks_perfectly():
    hw = ac.adaptcore_get_hw()
    recs = records(lambda c: c["predicted_s"])
    ev = cal.evaluate(recs, hw, False)
    assert ev["shapes"] == len(SHAPES)
    assert ev["top1"] == 1.0 and ev["regret_geomean"] == pytest.approx(1.0)


def test_regret_of_a_wrong_choice():
    """Make every shape's model choice measure 1.5x the fastest candidate:
    top-1 drops to 0 and the regret is exactly 1.5."""
    hw = ac.adaptcore_get_hw()
    picks = {}
    for M, N, K in SHAPES:
        cands = ac.adaptcore_candidates(M, N, K, BF16, 0)
        picks[(M, N, K)] = min(cands, key=lambda c: (c["predicted_s"], c["variant_key"]))["variant_key"]
    recs = records(lambda c: 2.0)
    for r in recs:
        if r["key"] == picks[(r["M"], r["N"], r["K"])]:
            r["t"] = 3.0
    ev = cal.evaluate(recs, hw, False)
    assert ev["top1"] == 0.0
    assert ev["regret_geomean"] == pytest.approx(1.5) and ev["regret_max"] == pytest.approx(1.5)
    assert math.isclose(ev["within_10pct"], 0.0)


def test_splice_replaces_one_family_on_the_remeasured_shapes(tmp_path):
    import json
    old = [dict(M=1, N=2, K=3, dtype=BF16, family="direct", key=1, t=1.0),
           dict(M=1, N=2, K=3, dtype=BF16, family="tile", key=2, t=2.0),
           dict(M=4, N=5, K=6, dtype=BF16, family="direct", key=1, t=3.0)]
    new = [dict(M=1, N=2, K=3, dtype=BF16, family="direct", key=1, t=0.5),
           dict(M=1, N=2, K=3, dtype=BF16, family="direct", key=3, t=0.7)]
    paths = [tmp_path / n for n in ("old.json", "new.json", "out.json")]
    for p, recs in zip(paths, (old, new)):
        p.write_text(json.dumps(recs))
    cal.main(["splice"] + [str(p) for p in paths])
    out = json.loads(paths[2].read_text())
    got = sorted((r["M"], r["family"], r["key"], r["t"]) for r in out)
    assert got == [(1, "direct", 1, 0.5), (1, "direct", 3, 0.7), (1, "tile", 2, 2.0), (4, "direct", 1, 3.0)]


def test_family_refit_holds_the_rest_of_the_profile():
    """Time one family's candidates at three times the model's price: a
    refit of that family alone lowers the loss and leaves the global
    constants and every other configuration's constants as they were."""
    hw = ac.adaptcore_get_hw()
    fam = "direct"
    recs = records(lambda c: c["predicted_s"] * (3.0 if c["family_name"] == fam else 1.0))
    only = {cal.config_of(r["key"]) for r in recs if r["family"] == fam}
    assert only
    h, stats = cal.fit(recs, hw, log=lambda m: None, only=only)
    assert stats["loss_after"] < stats["loss_before"]
    for name in cal.FIT_FIELDS:
        assert getattr(h, name) == getattr(hw, name), name
    for i in range(ac.AC_N_CFG):
        if i not in only:
            assert (h.cfg_iter[i], h.cfg_wg[i], h.cfg_wr[i]) == (hw.cfg_iter[i], hw.cfg_wg[i], hw.cfg_wr[i]), i
    assert any(h.cfg_iter[i] != hw.cfg_iter[i] or h.cfg_wg[i] != hw.cfg_wg[i] for i in only)
