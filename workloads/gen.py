"""Seeded input generators (numpy only).

Shape sets
  single_512()       one 512^3 product, fp32 output
  skinny_m()         decode-style products: M in {1..64} x (N, K) in
                     {(4096,4096), (14336,4096), (4096,14336)}, bf16 output
  small_mn_large_k() (M, N) in {(64,64), (128,256), (512,512)} x
                     K in {65536, 131072, 262144}, fp32 output
  sweep(n, seed)     dynamic-shape sweep: M, N, K log-uniform integers in
                     [1, 100000], a triple rejected if M*N*K > 2^37 or any
                     operand (A, B, bf16 C) exceeds 4 GiB
  moe_counts(...)    per-step token counts of 8192 tokens routed over 64
                     experts with Zipf(1.2)-distributed loads

Values
  bf16_bits(x)       fp32 -> bf16 bit patterns, round to nearest even
  uniform_bf16(...)  i.i.d. uniform[-1, 1] rounded to bf16
  normal_bf16(...)   i.i.d. normal(0, sigma) rounded to bf16
  int_bf16(...)      i.i.d. integers in [-lim, lim] (exact in bf16)

The industrial shape set and the recommendation-model workloads of the
paper's evaluation are not public; these synthetic sets stand in for them.
"""
import math

import numpy as np

U16 = np.uint16


def bf16_bits(x):
    """fp32 array -> uint16 bf16 bit patterns, round to nearest, ties to even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    bias = ((u >> 16) & 1) + 0x7FFF
    out = ((u + bias) >> 16).astype(U16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def f16_bits(x):
    """fp32 array -> uint16 IEEE fp16 bit patterns, round to nearest, ties to even."""
    return np.ascontiguousarray(x, dtype=np.float32).astype(np.float16).view(U16)


def uniform_f16(rows, cols, seed, lo=-1.0, hi=1.0):
    rng = np.random.default_rng(seed)
    return f16_bits(rng.uniform(lo, hi, size=(rows, cols)).astype(np.float32))


def uniform_bf16(rows, cols, seed, lo=-1.0, hi=1.0):
    rng = np.random.default_rng(seed)
    return bf16_bits(rng.uniform(lo, hi, size=(rows, cols)).astype(np.float32))


def normal_bf16(rows, cols, seed, sigma=1.0):
    rng = np.random.default_rng(seed)
    return bf16_bits((rng.standard_normal(size=(rows, cols)) * sigma).astype(np.float32))


def int_bf16(rows, cols, seed, lim=4):
    rng = np.random.default_rng(seed)
    return bf16_bits(rng.integers(-lim, lim + 1, size=(rows, cols)).astype(np.float32))


def uniform_f32(rows, cols, seed, lo=-1.0, hi=1.0):
    """fp32 values (an AddMM input C or bias row)."""
    rng = np.random.default_rng(seed)
    return rng.uniform(lo, hi, size=(rows, cols)).astype(np.float32)


def operands(M, N, K, seed, dist="uniform"):
    """A (M x K) and B (K x N) bf16 bit patterns for one shape ("uniform_f16":
    fp16 bit patterns of the same distribution)."""
    if dist == "uniform_f16":
        return uniform_f16(M, K, (seed, 0)), uniform_f16(K, N, (seed, 1))
    if dist == "uniform":
        return uniform_bf16(M, K, (seed, 0)), uniform_bf16(K, N, (seed, 1))
    if dist == "normal":  # normal(0, 1/sqrt(K)), sigma read as the std
        s = 1.0 / math.sqrt(max(K, 1))
        return normal_bf16(M, K, (seed, 0), s), normal_bf16(K, N, (seed, 1), s)
    if dist == "int":
        return int_bf16(M, K, (seed, 0)), int_bf16(K, N, (seed, 1))
    raise ValueError(dist)


# ---- shape sets ---------------------------------------------------------

def single_512():
    return [(512, 512, 512)]


def skinny_m():
    return [(m, n, k) for (n, k) in ((4096, 4096), (14336, 4096), (4096, 14336))
            for m in (1, 2, 4, 8, 16, 32, 64)]


def small_mn_large_k():
    return [(m, n, k) for (m, n) in ((64, 64), (128, 256), (512, 512))
            for k in (65536, 131072, 262144)]


SWEEP_MAX_DIM = 100000
SWEEP_MAX_MNK = 2 ** 37
SWEEP_MAX_OPERAND = 4 * 2 ** 30


def sweep_accepts(M, N, K):
    return (M * N * K <= SWEEP_MAX_MNK and 2 * M * K <= SWEEP_MAX_OPERAND
            and 2 * K * N <= SWEEP_MAX_OPERAND and 2 * M * N <= SWEEP_MAX_OPERAND)


def sweep(n=2000, seed=4, return_rejections=False):
    """Dynamic-shape sweep.

    Each dimension is round(exp(u)) clamped to [1, 100000], u ~ U[0, ln 1e5],
    drawn from numpy's PCG64 stream `default_rng(seed)` in the order M, N, K.
    A triple that breaks a size limit is rejected and redrawn as a whole.
    """
    rng = np.random.default_rng(seed)
    hi = math.log(SWEEP_MAX_DIM)
    out, rej = [], 0
    while len(out) < n:
        u = rng.uniform(0.0, hi, size=3)
        M, N, K = (min(max(int(round(math.exp(v))), 1), SWEEP_MAX_DIM) for v in u)
        if sweep_accepts(M, N, K):
            out.append((M, N, K))
        else:
            rej += 1
    return (out, rej) if return_rejections else out


def moe_counts(steps=100, tokens=8192, experts=64, s=1.2, seed=5, reading="B"):
    """Token counts per expert for each routing step (list of int arrays).

    Reading B (primary): each expert draws an i.i.d. Zipf(s) weight
    (numpy's zipf), weights are normalised and the tokens are multinomial.
    Reading A: a bounded rank-Zipf over the experts, p_r ~ r^-s, permuted
    every step, tokens multinomial.
    """
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(steps):
        if reading == "B":
            w = rng.zipf(s, size=experts).astype(np.float64)
        elif reading == "A":
            w = np.arange(1, experts + 1, dtype=np.float64) ** (-s)
            w = w[rng.permutation(experts)]
        else:
            raise ValueError(reading)
        p = w / w.sum()
        out.append(rng.multinomial(tokens, p).astype(np.int64))
    return out


MOE_HIDDEN = 4096
MOE_FFN = 1536


def moe_shapes(counts):
    """The per-expert GEMM calls of one routing step: up-projection
    (c x 4096) * (4096 x 1536), then down-projection (c x 1536) * (1536 x 4096)."""
    calls = []
    for e, c in enumerate(counts):
        calls.append((e, "up", int(c), MOE_FFN, MOE_HIDDEN))
        calls.append((e, "down", int(c), MOE_HIDDEN, MOE_FFN))
    return calls
