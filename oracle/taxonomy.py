"""Oracle for the planner arithmetic (test infrastructure only).

Plain, exact (rational) restatements of the paper's tiling taxonomy and the
closed forms of its performance model, each function citing the passage it
follows. The GPU library's planner implements the same quantities in its own
C++ code; tests compare the two. Nothing here is imported by the product.

Notation (paper Table 1, Section 4.2): the shape is (M, N, K); one core's
sub-task is m x n x k; an L1 tile is m1 x n1 x k1; task counts are
P_m = ceil(M/m), P_n = ceil(N/n), P_k = ceil(K/k).
"""
from fractions import Fraction

COMMON = "Common"
SINGLE = "SingleCoreSplitK"
MULTI = "MultiCoreSplitK"
HYBRID = "HybridSplitK"


def ceil_div(a, b):
    return -(-a // b)


def task_counts(M, N, K, m, n, k):
    """P_m, P_n, P_k (paper Table 1)."""
    return ceil_div(M, m), ceil_div(N, n), ceil_div(K, k)


def acc_tile_bytes(m1, n1, acc_bytes=4):
    """Bytes of the m1 x n1 accumulation tile in fp32 (Section 4.1)."""
    return m1 * n1 * acc_bytes


def classify(M, N, m, n, m1, n1, n_core, s_acc, acc_bytes=4):
    """Quadrant of the 2D template space (Section 4.2, the four templates).

    X axis: spatial sufficiency, P_m * P_n >= N_core.
    Y axis: on-chip accumulation, m1 * n1 * 4 B <= S_L0C.
    """
    pm, pn = ceil_div(M, m), ceil_div(N, n)
    spatial = pm * pn >= n_core
    on_chip = acc_tile_bytes(m1, n1, acc_bytes) <= s_acc
    if spatial and on_chip:
        return COMMON
    if spatial:
        return SINGLE
    if on_chip:
        return MULTI
    return HYBRID


def read_volume(M, N, K, m1, n1, elem_bytes=2):
    """Eq. 1: D_r = 2 * M*N*K * (1/m1 + 1/n1) bytes (fp16 inputs, no
    cross-tile residency). Exact rational value."""
    return Fraction(elem_bytes * M * N * K) * (Fraction(1, m1) + Fraction(1, n1))


def write_volume_common(M, N, out_bytes=2):
    """Eq. 2: each output written once after one cast."""
    return out_bytes * M * N


def write_volume_single(M, N, K, k1, out_bytes=2, acc_bytes=4):
    """Eq. 3: fp32 partials flushed after every k1 slice, plus the final cast."""
    return acc_bytes * M * N * ceil_div(K, k1) + out_bytes * M * N


def write_volume_multi(M, N, K, k, out_bytes=2, acc_bytes=4):
    """Eq. 4: one fp32 partial per K partition, plus the final cast."""
    return acc_bytes * M * N * ceil_div(K, k) + out_bytes * M * N


def write_volume_hybrid(M, N, K, k, k1, out_bytes=2, acc_bytes=4):
    """Eq. 5: P_k partitions, each flushing one fp32 partial of the whole
    M x N output after every k1 slice, plus the final cast.

    The printed left-hand side charges every partition ceil(k/k1) flushes; the
    last partition of a K that k does not divide is shorter, and is counted
    here with its actual length (Section 5.2 evaluates boundary tiles and the
    last K slice with their actual dimensions). Both sides of Eq. 5 equal this
    sum when k divides K and k1 divides k."""
    total = 0
    for p0 in range(0, K, k):
        total += acc_bytes * M * N * ceil_div(min(k, K - p0), k1)
    return total + out_bytes * M * N


def write_volume(cls, M, N, K, k, k1, out_bytes=2, acc_bytes=4):
    if cls == COMMON:
        return write_volume_common(M, N, out_bytes)
    if cls == SINGLE:
        return write_volume_single(M, N, K, k1, out_bytes, acc_bytes)
    if cls == MULTI:
        return write_volume_multi(M, N, K, k, out_bytes, acc_bytes)
    return write_volume_hybrid(M, N, K, k, k1, out_bytes, acc_bytes)


# --- Section 5.2 / 5.3: latency model ------------------------------------

def resource_cost(n_instr, lam, nbytes, bw, eta):
    """Eq. 8: t = n * lambda + D / (BW * eta)."""
    return Fraction(n_instr) * Fraction(lam) + Fraction(nbytes) / (Fraction(bw) * Fraction(eta))


def initiation_interval(stage_times, delta_dep=0):
    """Eq. 9: II = max over recurring stages + exposed dependency latency."""
    return max(Fraction(t) for t in stage_times) + Fraction(delta_dep)


def main_loop(tiles):
    """Eq. 10: sum over a core's tiles of T_fill + (L_v - 1) * II_v + T_drain.
    `tiles` is a sequence of (T_fill, L_v, II_v, T_drain)."""
    return sum((Fraction(f) + (L - 1) * Fraction(ii) + Fraction(d) for f, L, ii, d in tiles),
               Fraction(0))


def total_latency(t_pro, per_core_main, t_epi):
    """Eq. 7: T = T_pro + max over participating cores of T_main + T_epi."""
    return Fraction(t_pro) + max(Fraction(t) for t in per_core_main) + Fraction(t_epi)


def epilogue(t_local_reduce=0, t_cross_reduce=0, t_format=0):
    """Eq. 11."""
    return Fraction(t_local_reduce) + Fraction(t_cross_reduce) + Fraction(t_format)


def t_baseline(L, tM, tP, t_drain):
    """Eq. 12: one buffer, so loads and compute alternate."""
    return L * (Fraction(tM) + Fraction(tP)) + Fraction(t_drain)


def t_double_buffer(L, tM, tP, t_drain):
    """Eq. 13: two buffers, slices issued every max(t_M, t_P) after the fill."""
    tM, tP = Fraction(tM), Fraction(tP)
    return tM + (L - 1) * max(tM, tP) + tP + Fraction(t_drain)


def t_preload(Q, L, tM, tP, t_drain):
    """Eq. 14: Q regular tiles on one core with the first load of each tile
    advanced into the previous tile; every tile still pays its drain."""
    tM, tP = Fraction(tM), Fraction(tP)
    return tM + (Q * L - 1) * max(tM, tP) + tP + Q * Fraction(t_drain)


def ii_baseline(tM, tP):
    """Initiation interval of the baseline schedule (Section 5.3)."""
    return Fraction(tM) + Fraction(tP)


def ii_double_buffer(tM, tP):
    """Initiation interval with double buffering (Section 5.3)."""
    return max(Fraction(tM), Fraction(tP))
