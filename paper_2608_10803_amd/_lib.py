"""ctypes binding of libadaptcore.so: argument marshalling only.

Every function has the name and argument order of the C entry point in
include/adaptcore.h. Device memory and streams are passed as integers
(addresses / hipStream_t handles); `torch` is optional and only used by the
convenience wrapper `matmul_tensors`. The library must be built
(`python -m paper_2608_10803_amd.build`); there is no fallback.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libadaptcore.so")

AC_N_CFG = 96  # calibrated cost table size (include/adaptcore.h)
AC_OK = 0
AC_ERR_INVALID_VALUE = -1
AC_ERR_UNSUPPORTED = -2
AC_ERR_OUT_OF_MEMORY = -3
AC_ERR_LAUNCH = -4
AC_ERR_NOT_INITIALIZED = -5
AC_ERR_INTERNAL = -6

AC_BF16_F32OUT = 0
AC_BF16_BF16OUT = 1
AC_F16_F32OUT = 2
AC_F16_F16OUT = 3
AC_FP16_F32OUT, AC_FP16_FP16OUT = AC_F16_F32OUT, AC_F16_F16OUT
AC_LAYOUT_ROW_ROW = 0
AC_LAYOUT_A_COL = 1  # A stored column-major (lda >= M)
AC_LAYOUT_B_COL = 2  # B stored column-major (ldb >= K)
AC_LAYOUT_COL_COL = 3
AC_A_ROWMAJOR, AC_A_COLMAJOR, AC_B_ROWMAJOR, AC_B_COLMAJOR = 0, AC_LAYOUT_A_COL, 0, AC_LAYOUT_B_COL
(AC_FAMILY_TILE, AC_FAMILY_SKINNY_M, AC_FAMILY_SKINNY_N, AC_FAMILY_STREAMK, AC_FAMILY_SMALLK, AC_FAMILY_DIRECT,
 AC_FAMILY_GROUPED, AC_FAMILY_PERSIST, AC_FAMILY_BATCHED, AC_FAMILY_DL, AC_FAMILY_TALL, AC_FAMILY_DL_OFFCHIP) = range(12)

CLASS_NAMES = ["Common", "SingleCoreSplitK", "MultiCoreSplitK", "HybridSplitK"]
FAMILY_NAMES = ["tile", "skinny_m", "skinny_n", "streamk", "smallk", "direct", "grouped", "persist", "batched", "dl",
                "tall", "offchip"]


class AdaptCoreError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("adaptcore error %d: %s" % (status, msg))
        self.status = status


class PlanDesc(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int64), ("N", ctypes.c_int64), ("K", ctypes.c_int64),
                ("dtype", ctypes.c_int32), ("layouts", ctypes.c_uint32),
                ("shape_key", ctypes.c_uint64), ("variant_key", ctypes.c_uint64),
                ("cls", ctypes.c_int32), ("family", ctypes.c_int32),
                ("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32), ("tile_k", ctypes.c_int32),
                ("pm", ctypes.c_int32), ("pn", ctypes.c_int32), ("pk", ctypes.c_int32),
                ("grid_x", ctypes.c_int32), ("grid_y", ctypes.c_int32),
                ("swizzle", ctypes.c_int32), ("n_candidates", ctypes.c_int32),
                ("predicted_s", ctypes.c_double), ("workspace_bytes", ctypes.c_int64),
                ("groups", ctypes.c_int64)]

    def as_dict(self):
        d = {f: getattr(self, f) for f, _ in self._fields_}
        d["cls_name"] = CLASS_NAMES[self.cls]
        d["family_name"] = FAMILY_NAMES[self.family]
        return d


class Candidate(ctypes.Structure):
    _fields_ = [("variant_key", ctypes.c_uint64), ("cls", ctypes.c_int32), ("family", ctypes.c_int32),
                ("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32), ("tile_k", ctypes.c_int32),
                ("pk", ctypes.c_int32), ("grid_x", ctypes.c_int32), ("grid_y", ctypes.c_int32),
                ("predicted_s", ctypes.c_double)]

    def as_dict(self):
        d = {f: getattr(self, f) for f, _ in self._fields_}
        d["family_name"] = FAMILY_NAMES[self.family]
        return d


class Stats(ctypes.Structure):
    _fields_ = [("lookups", ctypes.c_uint64), ("hits", ctypes.c_uint64), ("misses", ctypes.c_uint64),
                ("entries", ctypes.c_uint64), ("launches", ctypes.c_uint64),
                ("miss_seconds", ctypes.c_double), ("class_count", ctypes.c_uint64 * 4)]


class Hw(ctypes.Structure):
    _fields_ = [("n_cu", ctypes.c_int32), ("lds_bytes", ctypes.c_int32), ("s_acc_bytes", ctypes.c_int64),
                ("clock_hz", ctypes.c_double), ("hbm_bw", ctypes.c_double), ("hbm_eta", ctypes.c_double),
                ("l2_bw_cu", ctypes.c_double), ("t_launch", ctypes.c_double),
                ("t_mem_latency", ctypes.c_double), ("t_wg", ctypes.c_double), ("mfma_eta", ctypes.c_double),
                ("lds_bw_cu", ctypes.c_double), ("unaligned_eta", ctypes.c_double), ("l2_hit", ctypes.c_double),
                ("search_open", ctypes.c_int32), ("enable_streamk", ctypes.c_int32),
                ("cfg_iter", ctypes.c_double * AC_N_CFG), ("cfg_wg", ctypes.c_double * AC_N_CFG),
                ("cfg_wr", ctypes.c_double * AC_N_CFG), ("swizzle_gain", ctypes.c_double)]

    def as_dict(self):
        d = {}
        for f, _ in self._fields_:
            v = getattr(self, f)
            d[f] = list(v) if f in ("cfg_iter", "cfg_wg", "cfg_wr") else v
        return d

    def copy(self):
        h = Hw()
        ctypes.memmove(ctypes.byref(h), ctypes.byref(self), ctypes.sizeof(Hw))
        return h


class TaxIn(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("M", "N", "K", "m", "n", "k", "m1", "n1", "k1", "n_core", "s_acc")] + \
               [("elem_bytes", ctypes.c_int32), ("out_bytes", ctypes.c_int32)]


class TaxOut(ctypes.Structure):
    _fields_ = [("pm", ctypes.c_int64), ("pn", ctypes.c_int64), ("pk", ctypes.c_int64), ("cls", ctypes.c_int32),
                ("acc_bytes", ctypes.c_int64), ("read_bytes", ctypes.c_double), ("write_bytes", ctypes.c_double)]


_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libadaptcore.so is not built: run `python -m paper_2608_10803_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        i64, i32, u32, u64, p, d = (ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64,
                                    ctypes.c_void_p, ctypes.c_double)
        L.adaptcore_init.argtypes = []
        L.adaptcore_init.restype = i32
        L.adaptcore_plan.argtypes = [i64, i64, i64, i32, u32]
        L.adaptcore_plan.restype = p
        L.adaptcore_plan_variant.argtypes = [i64, i64, i64, i32, u32, u64]
        L.adaptcore_plan_variant.restype = p
        L.adaptcore_set_override.argtypes = [u64]
        L.adaptcore_set_override.restype = i32
        L.adaptcore_get_override.argtypes = []
        L.adaptcore_get_override.restype = u64
        L.adaptcore_matmul.argtypes = [p, p, i64, p, i64, p, i64, p]
        L.adaptcore_matmul.restype = i32
        L.adaptcore_matmul_noalloc.argtypes = [p, p, i64, p, i64, p, i64, p]
        L.adaptcore_matmul_noalloc.restype = i32
        L.adaptcore_noalloc_scratch_bytes.argtypes = []
        L.adaptcore_noalloc_scratch_bytes.restype = i64
        L.adaptcore_addmm.argtypes = [p, p, i64, p, i64, p, i64, ctypes.c_float, ctypes.c_float, p, p]
        L.adaptcore_addmm.restype = i32
        L.adaptcore_grouped_plan.argtypes = [i64, i64, i64, i64, i32, u32]
        L.adaptcore_grouped_plan.restype = p
        L.adaptcore_grouped_plan_variant.argtypes = [i64, i64, i64, i64, i32, u32, u64]
        L.adaptcore_grouped_plan_variant.restype = p
        L.adaptcore_grouped_matmul.argtypes = [p, p, p, i64, p, i64, i64, p, i64, p]
        L.adaptcore_grouped_matmul.restype = i32
        L.adaptcore_batched_plan.argtypes = [i64, i64, i64, i64, i32, u32]
        L.adaptcore_batched_plan.restype = p
        L.adaptcore_batched_plan_variant.argtypes = [i64, i64, i64, i64, i32, u32, u64]
        L.adaptcore_batched_plan_variant.restype = p
        L.adaptcore_batched_matmul.argtypes = [p, p, i64, i64, p, i64, i64, p, i64, i64, p]
        L.adaptcore_batched_matmul.restype = i32
        L.adaptcore_batched_addmm.argtypes = [p, p, i64, i64, p, i64, i64, p, i64, i64, ctypes.c_float,
                                              ctypes.c_float, p, p]
        L.adaptcore_batched_addmm.restype = i32
        L.adaptcore_grouped_addmm.argtypes = [p, p, p, i64, p, i64, i64, p, i64, ctypes.c_float, ctypes.c_float, p,
                                              i64, p]
        L.adaptcore_grouped_addmm.restype = i32
        L.adaptcore_reserve_workspace.argtypes = [p, i64]
        L.adaptcore_reserve_workspace.restype = i32
        L.adaptcore_plan_info.argtypes = [p, ctypes.POINTER(PlanDesc)]
        L.adaptcore_plan_info.restype = i32
        L.adaptcore_plan_kernels.argtypes = [p, ctypes.c_char_p, i64]
        L.adaptcore_plan_kernels.restype = i32
        L.adaptcore_candidates.argtypes = [i64, i64, i64, i32, u32, ctypes.POINTER(Candidate), i64]
        L.adaptcore_candidates.restype = i64
        L.adaptcore_get_hw.argtypes = [ctypes.POINTER(Hw)]
        L.adaptcore_get_hw.restype = i32
        L.adaptcore_set_hw.argtypes = [ctypes.POINTER(Hw)]
        L.adaptcore_set_hw.restype = i32
        L.adaptcore_stats.argtypes = [ctypes.POINTER(Stats)]
        L.adaptcore_stats.restype = i32
        L.adaptcore_cache_clear.argtypes = []
        L.adaptcore_cache_clear.restype = i32
        L.adaptcore_bench_lookup.argtypes = [i64, i64, ctypes.POINTER(d)]
        L.adaptcore_bench_lookup.restype = i32
        L.adaptcore_read_probe.argtypes = [p, i64, p, p]
        L.adaptcore_read_probe.restype = i32
        L.adaptcore_last_error.argtypes = []
        L.adaptcore_last_error.restype = ctypes.c_char_p
        L.adaptcore_last_status.argtypes = []
        L.adaptcore_last_status.restype = i32
        L.adaptcore_taxonomy.argtypes = [ctypes.POINTER(TaxIn), ctypes.POINTER(TaxOut)]
        L.adaptcore_taxonomy.restype = i32
        L.adaptcore_schedule.argtypes = [i32, i64, i64, d, d, d]
        L.adaptcore_schedule.restype = d
        L.adaptcore_config_index.argtypes = [i32, i32]
        L.adaptcore_config_index.restype = i32
        _lib = L
    return _lib


def adaptcore_last_error():
    return lib().adaptcore_last_error().decode()


last_error = adaptcore_last_error


def adaptcore_last_status():
    return lib().adaptcore_last_status()


def _check(status):
    if status != AC_OK:
        raise AdaptCoreError(status, last_error())
    return status


def adaptcore_init():
    return _check(lib().adaptcore_init())


def adaptcore_plan(M, N, K, dtype=AC_BF16_BF16OUT, layouts=AC_LAYOUT_ROW_ROW):
    """Cached plan handle (int) for the shape."""
    h = lib().adaptcore_plan(M, N, K, dtype, layouts)
    if not h:
        raise AdaptCoreError(adaptcore_last_status(), last_error())
    return h


def adaptcore_plan_variant(M, N, K, dtype, layouts, variant_key):
    h = lib().adaptcore_plan_variant(M, N, K, dtype, layouts, variant_key)
    if not h:
        raise AdaptCoreError(adaptcore_last_status(), last_error())
    return h


def adaptcore_set_override(variant_key_or_0):
    """Force the configuration of this thread's later adaptcore_plan calls (0 = none)."""
    return _check(lib().adaptcore_set_override(variant_key_or_0))


def adaptcore_get_override():
    return lib().adaptcore_get_override()


def adaptcore_matmul(plan, A, lda, B, ldb, C, ldc, stream=0):
    """C = A * B on `stream`; A, B, C are device addresses (ints)."""
    return _check(lib().adaptcore_matmul(plan, A, lda, B, ldb, C, ldc, stream))


def adaptcore_matmul_noalloc(plan, A, lda, B, ldb, C, ldc, stream=0):
    """adaptcore_matmul with the library's fixed device scratch as workspace
    (allocates nothing)."""
    return _check(lib().adaptcore_matmul_noalloc(plan, A, lda, B, ldb, C, ldc, stream))


def adaptcore_noalloc_scratch_bytes():
    return lib().adaptcore_noalloc_scratch_bytes()


def adaptcore_addmm(plan, A, lda, B, ldb, C, ldc, alpha=1.0, beta=0.0, bias=0, stream=0):
    """C = alpha * A * B + beta * C + bias on `stream`; A, B, C, bias are
    device addresses (ints), bias = 0 for none."""
    return _check(lib().adaptcore_addmm(plan, A, lda, B, ldb, C, ldc, alpha, beta, bias, stream))


def adaptcore_grouped_plan(rows, groups, N, K, dtype=AC_BF16_BF16OUT, layouts=AC_LAYOUT_ROW_ROW):
    """Cached grouped-product plan handle (int)."""
    h = lib().adaptcore_grouped_plan(rows, groups, N, K, dtype, layouts)
    if not h:
        raise AdaptCoreError(adaptcore_last_status(), last_error())
    return h


def adaptcore_grouped_plan_variant(rows, groups, N, K, dtype, layouts, variant_key):
    h = lib().adaptcore_grouped_plan_variant(rows, groups, N, K, dtype, layouts, variant_key)
    if not h:
        raise AdaptCoreError(adaptcore_last_status(), last_error())
    return h


def adaptcore_grouped_matmul(plan, counts, A, lda, B, ldb, stride_b, C, ldc, stream=0):
    """Grouped product on `stream`; counts, A, B, C are device addresses."""
    return _check(lib().adaptcore_grouped_matmul(plan, counts, A, lda, B, ldb, stride_b, C, ldc, stream))


def adaptcore_grouped_addmm(plan, counts, A, lda, B, ldb, stride_b, C, ldc, alpha=1.0, beta=0.0, bias=0,
                            stride_bias=0, stream=0):
    """Grouped product with the AddMM epilogue on `stream` (bias row of group
    g at bias + g * stride_bias floats; bias = 0 for none)."""
    return _check(lib().adaptcore_grouped_addmm(plan, counts, A, lda, B, ldb, stride_b, C, ldc, alpha, beta, bias,
                                                stride_bias, stream))


def adaptcore_batched_plan(batch, M, N, K, dtype=AC_BF16_BF16OUT, layouts=AC_LAYOUT_ROW_ROW):
    """Cached strided-batch plan handle (int)."""
    h = lib().adaptcore_batched_plan(batch, M, N, K, dtype, layouts)
    if not h:
        raise AdaptCoreError(adaptcore_last_status(), last_error())
    return h


def adaptcore_batched_plan_variant(batch, M, N, K, dtype, layouts, variant_key):
    h = lib().adaptcore_batched_plan_variant(batch, M, N, K, dtype, layouts, variant_key)
    if not h:
        raise AdaptCoreError(adaptcore_last_status(), last_error())
    return h


def adaptcore_batched_matmul(plan, A, lda, stride_a, B, ldb, stride_b, C, ldc, stride_c, stream=0):
    """Strided batched product on `stream`; A, B, C are device addresses."""
    return _check(lib().adaptcore_batched_matmul(plan, A, lda, stride_a, B, ldb, stride_b, C, ldc, stride_c, stream))


def adaptcore_batched_addmm(plan, A, lda, stride_a, B, ldb, stride_b, C, ldc, stride_c, alpha=1.0, beta=0.0, bias=0,
                            stream=0):
    """C_b = alpha * A_b B_b + beta * C_b + bias for every batch b on `stream`;
    A, B, C, bias are device addresses (bias = 0 for none)."""
    return _check(lib().adaptcore_batched_addmm(plan, A, lda, stride_a, B, ldb, stride_b, C, ldc, stride_c, alpha,
                                                beta, bias, stream))


def adaptcore_reserve_workspace(stream, nbytes):
    return _check(lib().adaptcore_reserve_workspace(stream, nbytes))


def adaptcore_plan_info(plan):
    d = PlanDesc()
    _check(lib().adaptcore_plan_info(plan, ctypes.byref(d)))
    return d.as_dict()


def adaptcore_plan_kernels(plan):
    """Kernels one call of the plan launches, in launch order."""
    buf = ctypes.create_string_buffer(512)
    _check(lib().adaptcore_plan_kernels(plan, buf, len(buf)))
    return buf.value.decode().split(";")


def adaptcore_candidates(M, N, K, dtype=AC_BF16_BF16OUT, layouts=AC_LAYOUT_ROW_ROW):
    n = lib().adaptcore_candidates(M, N, K, dtype, layouts, None, 0)
    if n < 0:
        raise AdaptCoreError(n, last_error())
    arr = (Candidate * max(n, 1))()
    lib().adaptcore_candidates(M, N, K, dtype, layouts, arr, n)
    return [arr[i].as_dict() for i in range(n)]


def adaptcore_get_hw():
    h = Hw()
    _check(lib().adaptcore_get_hw(ctypes.byref(h)))
    return h


def adaptcore_set_hw(h):
    return _check(lib().adaptcore_set_hw(ctypes.byref(h)))


def adaptcore_stats():
    s = Stats()
    _check(lib().adaptcore_stats(ctypes.byref(s)))
    d = {f: getattr(s, f) for f, _ in Stats._fields_ if f != "class_count"}
    d["class_count"] = list(s.class_count)
    return d


def adaptcore_cache_clear():
    return _check(lib().adaptcore_cache_clear())


def adaptcore_read_probe(buf, nbytes, sink, stream=0):
    """Measurement reference: read `nbytes` of the device buffer once."""
    return _check(lib().adaptcore_read_probe(buf, nbytes, sink, stream))


def adaptcore_bench_lookup(n_keys, n_lookups):
    out = ctypes.c_double()
    _check(lib().adaptcore_bench_lookup(n_keys, n_lookups, ctypes.byref(out)))
    return out.value


def adaptcore_taxonomy(M, N, K, m, n, k, m1, n1, k1, n_core, s_acc, elem_bytes=2, out_bytes=2):
    i = TaxIn(M, N, K, m, n, k, m1, n1, k1, n_core, s_acc, elem_bytes, out_bytes)
    o = TaxOut()
    _check(lib().adaptcore_taxonomy(ctypes.byref(i), ctypes.byref(o)))
    return {"pm": o.pm, "pn": o.pn, "pk": o.pk, "cls": CLASS_NAMES[o.cls], "acc_bytes": o.acc_bytes,
            "read_bytes": o.read_bytes, "write_bytes": o.write_bytes}


def adaptcore_config_index(family, cfg):
    return lib().adaptcore_config_index(family, cfg)


def adaptcore_schedule(kind, Q, L, t_m, t_p, t_drain):
    return lib().adaptcore_schedule(kind, Q, L, t_m, t_p, t_drain)


def _operand(t, rows, cols):
    """(column-major?, leading dimension) of a 2-D operand view: rows
    contiguous (stride(1) == 1) or columns contiguous (stride(0) == 1)."""
    if t.dim() != 2 or not t.is_cuda:
        raise ValueError("operands must be 2-D GPU tensors")
    if cols <= 1 or t.stride(1) == 1:
        col, ld, need = False, (t.stride(0) if rows > 1 else cols), cols
    elif rows <= 1 or t.stride(0) == 1:
        col, ld, need = True, (t.stride(1) if cols > 1 else rows), rows
    else:
        raise ValueError("operands must have contiguous rows or contiguous columns")
    if ld < need:
        raise ValueError("overlapping operand view")
    return col, max(ld, 1)


def _marshal_tensors(A, B, C):
    """(M, N, K, dtype code, layouts, lda, ldb, ldc) of a tensor product,
    after the checks. A and B may be transposed views (contiguous columns);
    C must have contiguous rows."""
    import torch
    M, K = A.shape
    K2, N = B.shape
    if K2 != K or tuple(C.shape) != (M, N):
        raise ValueError("shape mismatch")
    if A.dtype != B.dtype or A.dtype not in (torch.bfloat16, torch.float16):
        raise TypeError("A and B must both be bfloat16 or both float16")
    f16 = A.dtype == torch.float16
    if C.dtype == torch.float32:
        dt = AC_F16_F32OUT if f16 else AC_BF16_F32OUT
    elif C.dtype == A.dtype:
        dt = AC_F16_F16OUT if f16 else AC_BF16_BF16OUT
    else:
        raise TypeError("C must be float32 or the input type")
    a_col, lda = _operand(A, M, K)
    b_col, ldb = _operand(B, K, N)
    if C.dim() != 2 or not C.is_cuda or (N > 1 and C.stride(1) != 1):
        raise ValueError("C must be a 2-D GPU tensor with contiguous rows")
    layouts = (AC_LAYOUT_A_COL if a_col else 0) | (AC_LAYOUT_B_COL if b_col else 0)
    return M, N, K, dt, layouts, lda, ldb, max(C.stride(0), N, 1)


def matmul_tensors(A, B, C, stream=None, plan=None):
    """C = A @ B for torch tensors on the GPU: 2-D, A and B with contiguous
    rows or contiguous columns (a transposed view selects the column-major
    layout), C with contiguous rows. A and B are both torch.bfloat16 or both
    torch.float16, C torch.float32 or the input type.
    Marshals pointers and leading dimensions; all arithmetic runs in the
    library's kernels."""
    import torch
    M, N, K, dt, layouts, lda, ldb, ldc = _marshal_tensors(A, B, C)
    if plan is None:
        plan = adaptcore_plan(M, N, K, dt, layouts)
    s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    adaptcore_matmul(plan, A.data_ptr(), lda, B.data_ptr(), ldb, C.data_ptr(), ldc, s)
    return C


def addmm_tensors(A, B, C, alpha=1.0, beta=0.0, bias=None, stream=None, plan=None):
    """C = alpha * A @ B + beta * C + bias in place, for torch tensors laid out
    as in matmul_tensors; bias is None or a contiguous float32 GPU tensor of
    N elements."""
    import torch
    M, N, K, dt, layouts, lda, ldb, ldc = _marshal_tensors(A, B, C)
    bp = 0
    if bias is not None:
        if bias.dtype != torch.float32 or bias.numel() != N or not bias.is_cuda or not bias.is_contiguous():
            raise ValueError("bias must be a contiguous float32 GPU tensor of N elements")
        bp = bias.data_ptr()
    if plan is None:
        plan = adaptcore_plan(M, N, K, dt, layouts)
    s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    adaptcore_addmm(plan, A.data_ptr(), lda, B.data_ptr(), ldb, C.data_ptr(), ldc, float(alpha), float(beta), bp, s)
    return C


def _dtype_code(A, B, C):
    import torch
    if A.dtype != B.dtype or A.dtype not in (torch.bfloat16, torch.float16):
        raise TypeError("A and B must both be bfloat16 or both float16")
    f16 = A.dtype == torch.float16
    if C.dtype == torch.float32:
        return AC_F16_F32OUT if f16 else AC_BF16_F32OUT
    if C.dtype == A.dtype:
        return AC_F16_F16OUT if f16 else AC_BF16_BF16OUT
    raise TypeError("C must be float32 or the input type")


def _rows_contiguous(t, name):
    if not t.is_cuda or (t.shape[-1] > 1 and t.stride(-1) != 1):
        raise ValueError("%s must be a GPU tensor with contiguous rows" % name)


def bmm_tensors(A, B, C, alpha=None, beta=0.0, bias=None, stream=None, plan=None):
    """C[b] = A[b] @ B[b] for 3-D torch tensors on the GPU (batch x M x K,
    batch x K x N, batch x M x N; contiguous rows, any batch stride, B may be
    broadcast with batch stride 0). With alpha given: C[b] = alpha * A[b] @
    B[b] + beta * C[b] + bias (bias None or N float32 values), in place.
    Marshals pointers, leading dimensions and strides only."""
    import torch
    batch, M, K = A.shape
    batch2, K2, N = B.shape
    if batch2 != batch or K2 != K or tuple(C.shape) != (batch, M, N):
        raise ValueError("shape mismatch")
    dt = _dtype_code(A, B, C)
    for t, n in ((A, "A"), (B, "B"), (C, "C")):
        _rows_contiguous(t, n)
    lda, ldb, ldc = max(A.stride(1), K, 1), max(B.stride(1), N, 1), max(C.stride(1), N, 1)
    if plan is None:
        plan = adaptcore_batched_plan(batch, M, N, K, dt)
    s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    if alpha is None:
        adaptcore_batched_matmul(plan, A.data_ptr(), lda, A.stride(0), B.data_ptr(), ldb, B.stride(0), C.data_ptr(),
                                 ldc, C.stride(0), s)
    else:
        bp = 0
        if bias is not None:
            if bias.dtype != torch.float32 or bias.numel() != N or not bias.is_cuda or not bias.is_contiguous():
                raise ValueError("bias must be a contiguous float32 GPU tensor of N elements")
            bp = bias.data_ptr()
        adaptcore_batched_addmm(plan, A.data_ptr(), lda, A.stride(0), B.data_ptr(), ldb, B.stride(0), C.data_ptr(),
                                ldc, C.stride(0), float(alpha), float(beta), bp, s)
    return C


def grouped_mm_tensors(A, B, counts, C, stream=None, plan=None):
    """The grouped product for torch tensors on the GPU: A (rows x K) holds
    the groups' rows one after another, B (groups x K x N, or K x N shared
    by all groups), counts an int32 GPU tensor of `groups` row counts (read by
    the kernel, never by the host), C (rows x N). Contiguous rows required.
    Marshals pointers, leading dimensions and strides only."""
    import torch
    rows, K = A.shape
    if B.dim() == 2:
        groups, stride_b = counts.numel(), 0
        K2, N = B.shape
        ldb = max(B.stride(0), N, 1)
    else:
        groups, K2, N = B.shape
        stride_b, ldb = B.stride(0), max(B.stride(1), N, 1)
    if K2 != K or tuple(C.shape) != (rows, N) or counts.numel() != groups:
        raise ValueError("shape mismatch")
    if counts.dtype != torch.int32 or not counts.is_cuda or not counts.is_contiguous():
        raise ValueError("counts must be a contiguous int32 GPU tensor")
    dt = _dtype_code(A, B, C)
    for t, n in ((A, "A"), (B, "B"), (C, "C")):
        _rows_contiguous(t, n)
    if plan is None:
        plan = adaptcore_grouped_plan(rows, groups, N, K, dt)
    s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    adaptcore_grouped_matmul(plan, counts.data_ptr(), A.data_ptr(), max(A.stride(0), K, 1), B.data_ptr(), ldb,
                             stride_b, C.data_ptr(), max(C.stride(0), N, 1), s)
    return C
