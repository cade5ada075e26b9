"""Pins for the planner oracle (CPU only).

* The four worked cases of Section 4.3 (printed task counts, accumulator
  bytes and template) from tests/golden/taxonomy_cases.json.
* Eq. 1 and Eqs. 2-5 against brute-force enumeration of tiles, slices and
  flushes on small shapes.
* Eqs. 12-13 against a discrete-event simulation of a load stage and a
  compute stage sharing one or two buffers; Eq. 14 against the same
  simulation where it is exact (compute-bound slices) and against Eq. 13 for a
  single tile.
"""
import itertools
import json
import os
from fractions import Fraction

import pytest

from oracle import taxonomy as tx

GOLD = os.path.join(os.path.dirname(__file__), "golden", "taxonomy_cases.json")


def load_cases():
    with open(GOLD) as f:
        return json.load(f)


@pytest.mark.parametrize("case", load_cases()["cases"], ids=lambda c: "case%d" % c["case"])
def test_paper_cases(case):
    g = load_cases()
    pm, pn, pk = tx.task_counts(case["M"], case["N"], case["K"], case["m"], case["n"], case["k"])
    assert pm * pn == case["tasks"]
    assert tx.acc_tile_bytes(case["m1"], case["n1"]) == case["acc_bytes"]
    assert tx.classify(case["M"], case["N"], case["m"], case["n"], case["m1"], case["n1"],
                       g["n_core"], g["s_acc"]) == case["class"]
    if "acc_bytes_before" in case:
        assert tx.acc_tile_bytes(case["m1_before"], case["n1_before"]) == case["acc_bytes_before"]
        # the smaller tile reads more (Eq. 1): enlarging is what reduces D_r
        assert (tx.read_volume(case["M"], case["N"], case["K"], case["m1"], case["n1"]) <
                tx.read_volume(case["M"], case["N"], case["K"], case["m1_before"], case["n1_before"]))
    if "idle_cores" in case:
        assert g["n_core"] - pm * pn == case["idle_cores"]


def enum_reads(M, N, K, m1, n1, k1, elem=2):
    """Bytes read when every L1 tile loads its m1 x k1 and k1 x n1 operand
    slices from memory (no reuse across tiles); M, N, K divisible by tiles."""
    total = 0
    for _i in range(0, M, m1):
        for _j in range(0, N, n1):
            for _k in range(0, K, k1):
                total += (m1 * k1 + k1 * n1) * elem
    return total


@pytest.mark.parametrize("M,N,K,m1,n1,k1", [(64, 32, 48, 16, 8, 16), (128, 128, 64, 32, 64, 32),
                                           (96, 160, 40, 32, 32, 8)])
def test_eq1_read_volume_by_enumeration(M, N, K, m1, n1, k1):
    assert tx.read_volume(M, N, K, m1, n1) == enum_reads(M, N, K, m1, n1, k1)


def enum_writes(M, N, K, m1, n1, k, k1, off_chip, out=2, acc=4):
    """Enumerate the writes of each template: for every K partition of length
    k and every output tile, either one fp32 export at the end of the
    partition (on-chip accumulation) or one fp32 flush after every k1 slice
    (off-chip); split K adds the partition exports; the final cast writes the
    output once."""
    total = 0
    parts = list(range(0, K, k))
    for _i in range(0, M, m1):
        for _j in range(0, N, n1):
            for p0 in parts:
                klen = min(k, K - p0)
                if off_chip:
                    total += m1 * n1 * acc * len(range(0, klen, k1))
                elif len(parts) > 1:
                    total += m1 * n1 * acc
    return total + M * N * out


@pytest.mark.parametrize("K,k,k1", [(64, 64, 16), (64, 16, 16), (70, 64, 16), (100, 30, 8),
                                    (96, 32, 32)])
def test_eqs2to5_write_volume_by_enumeration(K, k, k1):
    M, N, m1, n1 = 32, 48, 16, 16
    if k == K:
        assert tx.write_volume_common(M, N) == enum_writes(M, N, K, m1, n1, K, k1, False)
        assert tx.write_volume_single(M, N, K, k1) == enum_writes(M, N, K, m1, n1, K, k1, True)
    else:
        assert tx.write_volume_multi(M, N, K, k) == enum_writes(M, N, K, m1, n1, k, k1, False)
        assert tx.write_volume_hybrid(M, N, K, k, k1) == enum_writes(M, N, K, m1, n1, k, k1, True)
        if K % k == 0 and k % k1 == 0:  # the paper's equality in Eq. 5
            assert tx.write_volume_hybrid(M, N, K, k, k1) == tx.write_volume_single(M, N, K, k1)


def simulate(n_tiles, L, tM, tP, t_drain, buffers, carry_across_tiles):
    """Discrete-event simulation of a load unit and a compute unit.

    Slice s is loaded into buffer s % buffers; a load waits for the load unit
    and for the buffer's previous consumer; a compute waits for its load and
    for the compute unit. The drain of a tile runs on the compute unit after
    the tile's last slice. Without carry_across_tiles, a tile's first load
    waits until the previous tile has drained (double buffering per tile)."""
    load_free = Fraction(0)
    comp_free = Fraction(0)
    consumed = {}  # buffer -> time its last consumer finished
    s = 0
    for t in range(n_tiles):
        if not carry_across_tiles:
            load_free = max(load_free, comp_free)
            consumed = {b: comp_free for b in consumed}
        for _l in range(L):
            b = s % buffers
            start = max(load_free, consumed.get(b, Fraction(0)))
            load_end = start + tM
            load_free = load_end
            c_start = max(load_end, comp_free)
            comp_free = c_start + tP
            consumed[b] = comp_free
            s += 1
        comp_free += t_drain
    return comp_free


VALUES = [Fraction(x) for x in (1, 2, 3, Fraction(5, 2), 7)]


@pytest.mark.parametrize("L", [1, 2, 5])
def test_eq12_eq13_by_simulation(L):
    for tM, tP, td in itertools.product(VALUES, VALUES, [Fraction(0), Fraction(3, 2)]):
        assert tx.t_baseline(L, tM, tP, td) == simulate(1, L, tM, tP, td, 1, False)
        assert tx.t_double_buffer(L, tM, tP, td) == simulate(1, L, tM, tP, td, 2, False)
        # double buffering per tile, Q tiles in a row (the comparison in Section 5.3)
        assert 3 * tx.t_double_buffer(L, tM, tP, td) == simulate(3, L, tM, tP, td, 2, False)
        assert tx.ii_baseline(tM, tP) == tM + tP
        assert tx.ii_double_buffer(tM, tP) == max(tM, tP)


@pytest.mark.parametrize("Q,L", [(1, 3), (2, 2), (4, 3)])
def test_eq14_preload(Q, L):
    for tM, tP, td in itertools.product(VALUES, VALUES, [Fraction(0), Fraction(1, 2)]):
        if Q == 1:
            assert tx.t_preload(1, L, tM, tP, td) == tx.t_double_buffer(L, tM, tP, td)
        if tP >= tM:  # compute-bound: every drain sits on the critical path
            assert tx.t_preload(Q, L, tM, tP, td) == simulate(Q, L, tM, tP, td, 2, True)
        # preloading never loses against per-tile double buffering, and gains
        # one overlapped fill per extra tile
        assert (Q * tx.t_double_buffer(L, tM, tP, td) - tx.t_preload(Q, L, tM, tP, td)
                == (Q - 1) * min(tM, tP))


def test_eq10_reduces_to_eq13():
    """With T_fill = t_M + t_P and II = max(t_M, t_P) the main-loop sum of
    Eq. 10 for one tile equals the double-buffered schedule of Eq. 13."""
    for tM, tP, td in itertools.product(VALUES, VALUES, [Fraction(0), Fraction(2)]):
        for L in (1, 4):
            ii = tx.initiation_interval([tM, tP])
            assert tx.main_loop([(tM + tP, L, ii, td)]) == tx.t_double_buffer(L, tM, tP, td)


def test_eq7_slowest_core():
    assert tx.total_latency(1, [3, 9, 4], 2) == 12
    assert tx.epilogue(1, 2, 3) == 6
    assert tx.resource_cost(4, Fraction(1, 2), 1024, 256, Fraction(1, 2)) == 10
