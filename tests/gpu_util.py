"""Helpers of the GPU parity tests: device buffers with canaries, one call
through the C ABI, and comparison with the oracle."""
import numpy as np

import paper_2608_10803_amd as ac
from oracle import gemm_ref

F32_CANARY = np.float32(-1.2345678e30)
BF16_CANARY = np.uint16(0xFF7F)  # bf16 -3.39e38, never produced by the tests' inputs


def torch():
    import torch as t
    if not t.cuda.is_available():
        raise RuntimeError("GPU tests need a GPU")
    return t


def to_device(bits, ld=None, offset=0):
    """uint16 matrix -> device buffer (rows x ld) holding it; returns (tensor,
    address of element (0, 0)). `offset` shifts the start by that many
    elements (unaligned pointers)."""
    t = torch()
    rows, cols = bits.shape
    ld = cols if ld is None else ld
    host = np.zeros(rows * ld + offset + 8, np.uint16)
    if rows and cols:
        host[offset:offset + rows * ld].reshape(rows, ld)[:, :cols] = bits
    dev = t.from_numpy(host.view(np.int16)).to("cuda")
    return dev, dev.data_ptr() + 2 * offset


def fp32_out(dtype):
    return dtype in (ac.AC_BF16_F32OUT, ac.AC_F16_F32OUT)


def fmt_of(dtype):
    """Format of the inputs (and of a 16-bit output) of a dtype."""
    return "fp16" if dtype in (ac.AC_F16_F32OUT, ac.AC_F16_F16OUT) else "bf16"


class Out:
    """Output buffer of M x N with leading dimension ldc, a canary row above
    and below and canary columns beyond N."""

    def __init__(self, M, N, ldc, dtype):
        t = torch()
        self.M, self.N, self.ldc, self.dtype = M, N, ldc, dtype
        n = (M + 2) * ldc
        if fp32_out(dtype):
            self.host = np.full(n, F32_CANARY, np.float32)
            self.dev = t.from_numpy(self.host.copy()).to("cuda")
            self.addr = self.dev.data_ptr() + 4 * ldc
        else:
            self.host = np.full(n, BF16_CANARY, np.uint16)
            self.dev = t.from_numpy(self.host.view(np.int16).copy()).to("cuda")
            self.addr = self.dev.data_ptr() + 2 * ldc

    def fill(self, vals):
        """Sets the M x N interior (fp32 values, or 16-bit bit patterns) and
        keeps the canaries around it."""
        host = self.host.copy()
        w = host.reshape(self.M + 2, self.ldc)
        w[1:self.M + 1, :self.N] = vals
        t = torch()
        src = host if fp32_out(self.dtype) else host.view(np.int16)
        self.dev.copy_(t.from_numpy(src.copy()).to("cuda"))

    def read(self):
        """(values as fp64 M x N, canaries intact?)"""
        raw = self.dev.cpu().numpy()
        if fp32_out(self.dtype):
            full = raw.reshape(self.M + 2, self.ldc)
            vals = full[1:self.M + 1, :self.N].astype(np.float64)
            canary = F32_CANARY
        else:
            full = raw.view(np.uint16).reshape(self.M + 2, self.ldc)
            vals = gemm_ref.decode(np.ascontiguousarray(full[1:self.M + 1, :self.N]), fmt=fmt_of(self.dtype))
            canary = BF16_CANARY
        mask = np.ones(full.shape, bool)
        mask[1:self.M + 1, :self.N] = False
        ok = bool(np.all(full[mask] == canary))
        return vals, ok


def run(plan, A, B, M, N, K, dtype, lda=None, ldb=None, ldc=None, a_off=0, b_off=0, stream=0):
    """One adaptcore_matmul through the C ABI; returns (C values, canaries ok)."""
    t = torch()
    lda = max(K, 1) if lda is None else lda
    ldb = max(N, 1) if ldb is None else ldb
    ldc = max(N, 1) if ldc is None else ldc
    Ad, a = to_device(A, lda, a_off)
    Bd, b = to_device(B, ldb, b_off)
    out = Out(M, N, ldc, dtype)
    ac.adaptcore_matmul(plan, a, lda, b, ldb, out.addr, ldc, stream)
    t.cuda.synchronize()
    vals, ok = out.read()
    del Ad, Bd
    return vals, ok


def run_addmm(plan, A, B, M, N, K, dtype, c_old, alpha, beta, bias=None, lda=None, ldb=None, ldc=None,
              a_off=0, b_off=0, stream=0):
    """One adaptcore_addmm through the C ABI with C holding c_old (fp32
    values or 16-bit patterns) before the call; bias is None or N fp32
    values. Returns (C values, canaries ok)."""
    t = torch()
    lda = max(K, 1) if lda is None else lda
    ldb = max(N, 1) if ldb is None else ldb
    ldc = max(N, 1) if ldc is None else ldc
    Ad, a = to_device(A, lda, a_off)
    Bd, b = to_device(B, ldb, b_off)
    out = Out(M, N, ldc, dtype)
    out.fill(c_old)
    bd = None
    if bias is not None:
        bd = t.from_numpy(np.ascontiguousarray(bias, np.float32)).to("cuda")
    ac.adaptcore_addmm(plan, a, lda, b, ldb, out.addr, ldc, alpha, beta, bd.data_ptr() if bd is not None else 0,
                       stream)
    t.cuda.synchronize()
    vals, ok = out.read()
    del Ad, Bd, bd
    return vals, ok


def tol(dtype):
    if fp32_out(dtype):
        return gemm_ref.TOL["f32"]
    return gemm_ref.TOL[fmt_of(dtype)]


# fp16 output: rounding to nearest even has relative error <= 2^-11 in the
# normal range (inside the 1e-3 bar) but absolute error up to half the
# subnormal spacing, 2^-25, below 2^-14; differences within that are exact.
F16_SUBNORMAL_HALF_ULP = 2.0 ** -25


def check(vals, ok, A, B, dtype, ref=None, label=""):
    assert ok, "write outside C (canary overwritten) %s" % label
    C_ref, D = ref if ref is not None else gemm_ref.gemm(A, B, fmt=fmt_of(dtype))
    if dtype == ac.AC_F16_F16OUT:
        vals = np.where(np.abs(vals - C_ref) <= F16_SUBNORMAL_HALF_ULP, C_ref, vals)
    err = gemm_ref.err_metric(vals, C_ref, D)
    assert err <= tol(dtype), "err %.3g > %.3g %s" % (err, tol(dtype), label)
    return err


def all_candidates(M, N, K, dtype, layouts=0):
    """Every legal configuration of a shape, including stream-K and the
    configurations outside the taxonomy's template."""
    hw = ac.adaptcore_get_hw()
    h2 = ac.adaptcore_get_hw()
    h2.search_open = 1
    h2.enable_streamk = 1
    ac.adaptcore_set_hw(h2)
    try:
        return ac.adaptcore_candidates(M, N, K, dtype, layouts)
    finally:
        ac.adaptcore_set_hw(hw)


def forced_plan(M, N, K, dtype, key, layouts=0):
    """Plan for a configuration key (valid until the next profile change)."""
    return ac.adaptcore_plan_variant(M, N, K, dtype, layouts, key)
