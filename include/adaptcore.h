/*
 * adaptcore.h -- C ABI of the adaptive dynamic-shape GEMM library for AMD
 * Instinct MI355X (gfx950).
 *
 * The library computes C = A * B for dense matrices of arbitrary (M, N, K)
 * (also with an AddMM epilogue, and as grouped and strided batched products),
 * following "Adaptive Matrix Multiplication for Dynamic Shapes on Ascend
 * NPUs" (AdaptCore), re-designed for gfx950:
 *   - a shape is mapped to a template of the 2D tiling taxonomy (Section 4.2:
 *     spatial parallelism x accumulation regime, worked cases in Section 4.3);
 *   - a deterministic analytical latency model (Section 5.2, Eqs. 7-14)
 *     selects the tile and the optimisation modules (Table 2) among the legal
 *     candidates (Eq. 6);
 *   - the selected configuration is cached under a 64-bit key of the shape
 *     (Section 3.2, online phase: the TilingKey lookup), so a repeated shape
 *     dispatches in O(1).
 *
 * Conventions for every entry point:
 *   - All functions are extern "C", never throw, and report failure through
 *     the return code (or NULL); adaptcore_last_error() then returns a
 *     thread-local message describing the last failure of the calling thread.
 *   - Matrices are dense and row-major (plain products may declare A or B
 *     column-major, AC_LAYOUT_*), with leading dimensions in ELEMENTS.
 *     A is M x K (lda >= max(1, K)), B is K x N (ldb >= max(1, N)),
 *     C is M x N (ldc >= max(1, N)). Inputs are bf16 or fp16 (raw 16-bit
 *     storage); accumulation is always fp32; C is fp32 or 16-bit in the
 *     input format (round to nearest even) as the plan's dtype says.
 *   - A, B, C are device pointers owned by the caller; they must be aligned
 *     to their element size and must not overlap C.
 *   - The library is single-GPU: every call uses the HIP device current on
 *     the calling thread.
 */
#ifndef ADAPTCORE_H
#define ADAPTCORE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  AC_OK = 0,
  AC_ERR_INVALID_VALUE = -1,   /* bad dimension, leading dimension, pointer or key */
  AC_ERR_UNSUPPORTED = -2,     /* dtype / layout not provided by this build */
  AC_ERR_OUT_OF_MEMORY = -3,   /* workspace allocation failed */
  AC_ERR_LAUNCH = -4,          /* the HIP runtime rejected a launch */
  AC_ERR_NOT_INITIALIZED = -5, /* no GPU, or workspace missing under stream capture */
  AC_ERR_INTERNAL = -6
} adaptcore_status;

/* Element types: 16-bit inputs (A and B in the same format), fp32
 * accumulation, and the output type. */
typedef enum {
  AC_BF16_F32OUT = 0,  /* bf16 inputs, C is fp32 */
  AC_BF16_BF16OUT = 1, /* bf16 inputs, C is bf16, rounded to nearest even */
  AC_F16_F32OUT = 2,   /* fp16 inputs, C is fp32 */
  AC_F16_F16OUT = 3    /* fp16 inputs, C is fp16, rounded to nearest even */
} adaptcore_dtype;
/* The fp16 codes under their longer names. */
enum { AC_FP16_F32OUT = AC_F16_F32OUT, AC_FP16_FP16OUT = AC_F16_F16OUT };

/* Operand layouts of plain products (adaptcore_plan, adaptcore_matmul,
 * adaptcore_addmm), a bit set: AC_LAYOUT_A_COL = A stored column-major
 * (element (i, k) at A[i + k * lda], lda >= M), AC_LAYOUT_B_COL = B stored
 * column-major (element (k, j) at B[k + j * ldb], ldb >= K); clear bits mean
 * row-major (A[i * lda + k], lda >= K; B[k * ldb + j], ldb >= N). The matrix
 * C is always row-major. A column-major operand is copied into a row-major
 * copy in the plan's workspace by a prologue kernel before the main kernel
 * (the copy prologue of the paper's padding module, priced as T_pro in
 * Eq. 7), except a column-major B under the small-M kernel, which reads it
 * in place. Grouped and batched products take row-major operands only. */
enum { AC_LAYOUT_ROW_ROW = 0, AC_LAYOUT_A_COL = 1, AC_LAYOUT_B_COL = 2, AC_LAYOUT_COL_COL = 3 };
/* The same bits named per operand (A_ROWMAJOR | B_COLMAJOR, ...). */
enum { AC_A_ROWMAJOR = 0, AC_A_COLMAJOR = AC_LAYOUT_A_COL, AC_B_ROWMAJOR = 0, AC_B_COLMAJOR = AC_LAYOUT_B_COL };

/* Templates of the 2D tiling taxonomy (Section 4.2). */
typedef enum {
  AC_CLASS_COMMON = 0,             /* P_m*P_n >= N_core, accumulator on chip */
  AC_CLASS_SINGLE_CORE_SPLITK = 1, /* P_m*P_n >= N_core, accumulator spills  */
  AC_CLASS_MULTI_CORE_SPLITK = 2,  /* P_m*P_n <  N_core, accumulator on chip */
  AC_CLASS_HYBRID_SPLITK = 3       /* P_m*P_n <  N_core, accumulator spills  */
} adaptcore_class;

/* Kernel families of the variant space. */
typedef enum {
  AC_FAMILY_TILE = 0,     /* MFMA macro-tile kernel, P_k >= 1 */
  AC_FAMILY_SKINNY_M = 1, /* Small-M Copy module: B streamed once, M <= 64 */
  AC_FAMILY_SKINNY_N = 2, /* Small-M Copy by orientation: A streamed once, N <= 64 */
  AC_FAMILY_STREAMK = 3,  /* StreamK applied to the tile kernel */
  AC_FAMILY_SMALLK = 4,   /* K <= 16: rank-K update bound by writing C */
  AC_FAMILY_DIRECT = 5,   /* small problems: MFMA fragments straight from memory, no LDS */
  AC_FAMILY_GROUPED = 6,  /* the tile kernel over the groups of a grouped product */
  AC_FAMILY_PERSIST = 7,  /* persistent tile kernel: the next tile's first k-block is fetched
                             before the current tile's epilogue (K >= 8, N >= 8) */
  AC_FAMILY_BATCHED = 8,  /* the grouped kernel over a strided batch of equal shapes */
  AC_FAMILY_DL = 9,       /* tile kernel with operand tiles loaded straight into LDS through 2-5
                             stages (Multi-Buffer), 32- to 256-row tiles. Rows of A and B that
                             are not whole 16-byte chunks are copied zero-padded first (the
                             Padding module), or loaded through registers (VariantKey bit 13);
                             at run time, misaligned operands run the register-load form or the
                             same tiling on AC_FAMILY_TILE. With P_k > 1 the partials are summed
                             by the reduction kernel */
  AC_FAMILY_TALL = 10,    /* N <= 32, A row-major: A streamed from HBM once through a
                             direct-to-LDS pipeline of 64-k stages, B's transposed copy (a
                             prologue) beside it; K not a multiple of 8 takes the register-load
                             form (VariantKey bit 13); misaligned A at run time runs that form,
                             or the same product on AC_FAMILY_SKINNY_N */
  AC_FAMILY_DL_OFFCHIP = 11 /* off-chip accumulation (the SingleCoreSplitK and HybridSplitK
                             templates, Section 4.2, Eqs. 3 and 5): a workgroup owns a
                             512 x 256 super-tile (two 256 x 256 tiles of AC_FAMILY_DL, whose
                             fp32 accumulator, 512 KiB, exceeds the 256 KiB of registers) and,
                             for each k1 slice of K in turn, computes both halves and flushes
                             their partial sums to the workspace; the reduction kernel adds the
                             slices. VariantKey: cfg = DL configuration | log2(workgroups along
                             K) << 4 (0: SingleCoreSplitK, > 0: HybridSplitK), P_k = slices.
                             Offered in the two off-chip templates and in the open search */
} adaptcore_family;

typedef struct adaptcore_plan_s adaptcore_plan_t; /* opaque, owned by the library */

/* Description of a plan (adaptcore_plan_info). */
typedef struct {
  int64_t M, N, K;
  int32_t dtype;
  uint32_t layouts;
  uint64_t shape_key;   /* 64-bit key of the shape (cache index) */
  uint64_t variant_key; /* 64-bit key of the selected configuration */
  int32_t cls;          /* adaptcore_class of the taxonomy for this shape */
  int32_t family;       /* adaptcore_family of the selected kernel */
  int32_t tile_m, tile_n, tile_k; /* m1, n1, k1 (workgroup output tile, k granule) */
  int32_t pm, pn, pk;   /* task counts P_m, P_n, P_k of the selected kernel */
  int32_t grid_x, grid_y; /* launch grid (workgroups of 256 threads) */
  int32_t swizzle;      /* 1 = XCD-aware grouped tile order (ShuffleK analogue) */
  int32_t n_candidates; /* legal candidates the model compared */
  double predicted_s;   /* model latency of the selected configuration, seconds */
  int64_t workspace_bytes; /* per stream: fp32 partials, then row-major copies of column-major
                              operands */
  int64_t groups;       /* grouped plans: number of groups (M is the row capacity); batched
                           plans: batch count (M, N, K of every batch); else 0 */
} adaptcore_plan_desc_t;

/* One legal candidate of a shape (adaptcore_candidates). */
typedef struct {
  uint64_t variant_key;
  int32_t cls, family, tile_m, tile_n, tile_k, pk, grid_x, grid_y;
  double predicted_s;
} adaptcore_candidate_t;

/* Counters (adaptcore_stats). */
typedef struct {
  uint64_t lookups;       /* adaptcore_plan calls */
  uint64_t hits;          /* served from the cache */
  uint64_t misses;        /* planned (taxonomy + model) */
  uint64_t entries;       /* plans held by the cache */
  uint64_t launches;      /* kernels launched by adaptcore_matmul */
  double miss_seconds;    /* total host time spent planning misses */
  uint64_t class_count[4];/* misses per taxonomy class */
} adaptcore_stats_t;

/* Hardware profile used by the planner. Defaults describe one MI355X
 * (256 CUs, 160 KiB LDS per CU); adaptcore_init() replaces the CU count with
 * the device's. The latency constants are the model's lambda / eta / BW of
 * Eq. 8, calibrated on the device. */
/* Number of kernel configurations with calibrated costs (table size). */
#define AC_N_CFG 96

typedef struct {
  int32_t n_cu;          /* N_core: compute units */
  int32_t lds_bytes;     /* LDS per CU */
  int64_t s_acc_bytes;   /* accumulator capacity of one workgroup (S_L0C analogue) */
  double clock_hz;       /* shader clock */
  double hbm_bw;         /* peak HBM bandwidth, bytes/s */
  double hbm_eta;        /* achievable fraction of hbm_bw for streaming reads */
  double l2_bw_cu;       /* per-CU bandwidth for cache-resident reads, bytes/s */
  double t_launch;       /* launch + dispatch cost of one kernel, s */
  double t_mem_latency;  /* exposed latency of a workgroup's first load, s */
  double t_wg;           /* fixed cost of one workgroup (setup, epilogue issue), s */
  double mfma_eta;       /* achievable fraction of MFMA issue rate */
  double lds_bw_cu;      /* LDS bytes per second per CU */
  double unaligned_eta;  /* bandwidth factor for rows that are not 16-byte aligned */
  double l2_hit;         /* fraction of tile re-reads served by L2 / MALL */
  int32_t search_open;   /* 0: search inside the taxonomy's template (Eq. 6);
                            1: search every template (the exhaustive reading) */
  int32_t enable_streamk; /* 1: StreamK candidates take part in the search */
  /* Per kernel configuration (index: adaptcore_config_index), calibrated by
   * profiling: cost of one main-loop iteration of a workgroup that has its CU
   * to itself, excluding memory transfer (the non-memory initiation interval
   * of Eq. 9), and the fixed cost of a workgroup (prologue, first-load
   * latency and epilogue together). 0 = use the analytic estimate: MFMA issue
   * and LDS traffic for the iteration, t_wg plus t_mem_latency per dependent
   * load phase for the fixed cost. Each value must lie in [0, 1) seconds. */
  double cfg_iter[AC_N_CFG];
  double cfg_wg[AC_N_CFG];
  /* Per kernel configuration: achieved fraction of the streaming HBM rate
   * (hbm_bw * hbm_eta) for the bytes the configuration writes (C or fp32
   * partials) -- the per-variant efficiency of Eq. 8 applied to the output
   * traffic. 0 = not calibrated (read as 1); each value in [0, 1]. */
  double cfg_wr[AC_N_CFG];
  /* Time factor of the main kernel of a tile-family plan with the XCD-aware
   * tile order (swizzle = 1) against the plain order: the order changes
   * which tiles share an XCD's L2, and so the traffic efficiency (Eq. 8's
   * eta) of both re-reads and output writes. In (0, 1]; 1 = no effect. */
  double swizzle_gain;
} adaptcore_hw_t;

/* Index of a kernel configuration in adaptcore_hw_t::cfg_iter / cfg_wg, or -1
 * (for AC_FAMILY_DL and AC_FAMILY_TALL, cfg | 0x100 names the configuration's register-load
 * form, VariantKey bit 13, which has a slot of its own). */
int32_t adaptcore_config_index(int32_t family, int32_t cfg);

/* Optional: bind the library to the current HIP device and read its CU count.
 * Without it, planning uses the default MI355X profile. AC_ERR_NOT_INITIALIZED
 * when no device is present. */
adaptcore_status adaptcore_init(void);

/* The problem statement of Section 5.1: given an input shape s = (M, N, K),
 * choose the configuration x* = argmin over the legal candidates S(b(s)) of
 * the modelled latency T(s; theta(s), x) (Eq. 6), where b(s) is the template
 * the taxonomy of Section 4.2 assigns to s. Section 3.2 (online phase): the
 * shape is packed into a 64-bit key and looked up in the plan cache; only a
 * miss runs the offline steps (taxonomy, candidate enumeration, latency
 * model of Eqs. 7-14, arg-min with ties to the smaller VariantKey).
 *
 * Returns the cached plan for (M, N, K, dtype, layouts): dtype one of
 * adaptcore_dtype, layouts a set of AC_LAYOUT_* bits. The same arguments
 * always return the same pointer until adaptcore_cache_clear(); the plan is
 * owned by the library (never freed by the caller). M, N, K >= 0 and < 2^31.
 * NULL on invalid or unsupported arguments (see adaptcore_last_error /
 * adaptcore_last_status). Host-only: no GPU work beyond reading the
 * device's kernel occupancies once; safe from many threads at once. While
 * adaptcore_set_override holds a key on the calling thread, the call
 * returns that configuration instead (adaptcore_plan_variant) and leaves
 * the cache untouched. */
const adaptcore_plan_t* adaptcore_plan(int64_t M, int64_t N, int64_t K, int32_t dtype, uint32_t layouts);

/* Like adaptcore_plan, but with the configuration forced to `variant_key`
 * (one of the keys listed by adaptcore_candidates): one point x of the
 * candidate set S(b(s)) of Eq. 6 instead of the arg-min. For tests and the
 * exhaustive model-accuracy experiment of Section 6.6. The plan is owned by
 * the library (a map of its own, not the shape cache). NULL if the key is
 * not legal for the shape (AC_ERR_INVALID_VALUE). */
const adaptcore_plan_t* adaptcore_plan_variant(int64_t M, int64_t N, int64_t K, int32_t dtype,
                                               uint32_t layouts, uint64_t variant_key);

/* Forces the configuration of every later adaptcore_plan call made by the
 * CALLING THREAD to `variant_key_or_0` (0 restores the model's choice): the
 * override hook of the exhaustive search of Section 6.6, which times every
 * legal configuration of a shape through the unchanged adaptcore_plan /
 * adaptcore_matmul path. The setting is thread-local; other threads and the
 * shape cache are not affected. With an override set, adaptcore_plan returns
 * adaptcore_plan_variant(M, N, K, dtype, layouts, key), i.e. NULL with
 * AC_ERR_INVALID_VALUE for shapes the key is not legal for (a key also
 * fixes dtype and layouts). Always AC_OK. For tests and timing only. */
adaptcore_status adaptcore_set_override(uint64_t variant_key_or_0);

/* The calling thread's override key (0 = none). */
uint64_t adaptcore_get_override(void);

/* Largest leading dimension (exclusive, in elements) of A and B accepted by
 * adaptcore_matmul: the kernels address operand tiles with 32-bit byte
 * offsets from a row base. */
#define AC_MAX_LD (1LL << 23)

/* Runs a plan: C = A * B, asynchronously on `stream` (a hipStream_t; NULL is
 * the null stream). This is the online execution of Section 3.2: the cached
 * configuration's kernels are launched by its VariantKey (the registry of
 * compiled templates, Section 4.2 and Table 2); every template computes the
 * same mathematical product C[i][j] = sum_k A[i][k] * B[k][j] (Section 4.1),
 * in fp32, with only the fp32 summation order differing between them. Validates the leading dimensions against the plan's
 * shape and layouts (row-major A: lda >= K, column-major A: lda >= M;
 * row-major B: ldb >= N, column-major B: ldb >= K; ldc >= N; all >= 1:
 * AC_ERR_INVALID_VALUE; a row-major lda or ldb >= AC_MAX_LD, or K or N of a
 * copied operand with its row padded to 8 reaching AC_MAX_LD:
 * AC_ERR_UNSUPPORTED) and the pointer alignment (A, B: 2 bytes; C: its
 * element size). M == 0 or N == 0: nothing is launched. K == 0: C is set to
 * zero.
 * Split-K plans and plans with a column-major operand use a workspace owned by the library for this (device,
 * stream); it is allocated on the stream's first use (outside any stream
 * capture: under capture a missing workspace gives AC_ERR_NOT_INITIALIZED)
 * and grows monotonically: a larger buffer replaces it for later calls, and
 * the replaced one is kept (never freed) until the process ends, so graphs
 * captured earlier and calls already enqueued keep valid memory. Concurrent
 * calls on ONE stream are ordered by the stream; calls on different streams
 * use different workspaces. Errors: AC_ERR_OUT_OF_MEMORY (workspace),
 * AC_ERR_LAUNCH (the runtime rejected a kernel), AC_ERR_NOT_INITIALIZED (no
 * device, or a missing workspace under capture); nothing is launched then
 * except kernels of the same call that were already enqueued. */
adaptcore_status adaptcore_matmul(const adaptcore_plan_t* plan, const void* A, int64_t lda, const void* B,
                                  int64_t ldb, void* C, int64_t ldc, void* stream);

/* ---- No-allocation variant ---------------------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc. It runs a
 * plain plan exactly as adaptcore_matmul does (same kernels, same results
 * bit for bit), but the workspace (split-K partials, stream-K pieces,
 * row-major copies of column-major operands) is a fixed array of device
 * memory compiled into the library, adaptcore_noalloc_scratch_bytes() bytes
 * (64 MiB) on every GPU the library runs on, held until the process ends.
 * No call of this entry point allocates or frees device memory. The
 * caller still passes A, B and C; arguments and checks are those of
 * adaptcore_matmul, and a plan whose workspace_bytes exceed the array gives
 * AC_ERR_UNSUPPORTED (nothing launched). Every call on one GPU shares that
 * GPU's array, and the array keeps the last call's contents: no part of it
 * needs clearing (every byte a call reads was written earlier in the same
 * call), but calls that overlap in time on one GPU (different streams, or
 * the same graph replayed concurrently) race on it -- order them. */
adaptcore_status adaptcore_matmul_noalloc(const adaptcore_plan_t* plan, const void* A, int64_t lda, const void* B,
                                          int64_t ldb, void* C, int64_t ldc, void* stream);

/* Size in bytes of the per-GPU array used by adaptcore_matmul_noalloc. */
int64_t adaptcore_noalloc_scratch_bytes(void);

/* ---- AddMM ------------------------------------------------------------------
 * AddMM is one of the dense operators the paper replaces in its end-to-end
 * models beside MatMul (Section 6.5; operator scope, Section 7). It runs a
 * plain plan with an epilogue applied to every element of C at the final
 * store, in fp32, before the rounding to C's type:
 *
 *   C[i][j] = alpha * (A * B)[i][j] + beta * C_old[i][j] + bias[j]
 *
 * C_old is C's content before the call (read only when beta != 0, so C may
 * hold anything when beta == 0); bias is a device array of N fp32 values
 * (NULL: no bias term). Split-K and stream-K plans apply the epilogue once,
 * in the kernel that writes the final value. Arguments, validation, workspace
 * and stream semantics are those of adaptcore_matmul; in addition alpha and
 * beta must be finite and bias aligned to 4 bytes (AC_ERR_INVALID_VALUE).
 * K == 0 yields C = beta * C_old + bias. A, B and bias must not overlap C. */
adaptcore_status adaptcore_addmm(const adaptcore_plan_t* plan, const void* A, int64_t lda, const void* B,
                                 int64_t ldb, void* C, int64_t ldc, float alpha, float beta, const float* bias,
                                 void* stream);

/* ---- Grouped product (GroupMM) ---------------------------------------------
 * The paper replaces the grouped products of its end-to-end models (GroupMM,
 * Section 6.5; operator scope, Section 7) as well as plain ones, and names
 * MoE routing as a source of run-time shape changes (Section 2.2). Here a
 * grouped product computes, for g = 0 .. groups-1,
 *     C[rows of g] = A[rows of g] * B_g,
 * in the contiguous form an MoE layer has after sorting tokens by expert:
 *   - A (rows x K, lda) and C (rows x N, ldc) are row-major with the rows of
 *     group 0, then group 1, ...; `rows` is the row capacity of A and C;
 *   - group g owns counts[g] consecutive rows; `counts` is a DEVICE array of
 *     `groups` int32 values that the host never reads (no synchronisation),
 *     so every count array is given a meaning: a negative count is read as
 *     0, and rows at or past `rows` are dropped -- group g covers rows
 *     [min(P_{g-1}, rows), min(P_g, rows)), P_g the running sum of the
 *     non-negative counts;
 *   - B_g (K x N, ldb, row-major) starts stride_b elements after B_{g-1}
 *     (stride_b = 0: all groups share one B).
 * Rows covered by no group are not written. Inputs bf16, fp32 accumulation,
 * C fp32 or bf16 as the plan's dtype says. One kernel launch per call.
 *
 * Returns the cached plan for (rows, groups, N, K, dtype, layouts): rows, N,
 * K in [0, 2^31), groups in [0, 2^20]. The model prices the balanced split
 * of the rows (the counts are not known when planning). NULL on invalid or
 * unsupported arguments. Host-only. */
const adaptcore_plan_t* adaptcore_grouped_plan(int64_t rows, int64_t groups, int64_t N, int64_t K, int32_t dtype,
                                               uint32_t layouts);

/* Like adaptcore_grouped_plan with the configuration forced to variant_key
 * (family AC_FAMILY_GROUPED, P_k = 1, a tile configuration that has a
 * grouped kernel). For tests. NULL if the key is not legal. */
const adaptcore_plan_t* adaptcore_grouped_plan_variant(int64_t rows, int64_t groups, int64_t N, int64_t K,
                                                       int32_t dtype, uint32_t layouts, uint64_t variant_key);

/* Runs a grouped plan asynchronously on `stream`. counts: device pointer to
 * the plan's `groups` int32 counts, read by the kernel when it runs. A, B, C
 * device pointers (A, B 2-byte aligned, C aligned to its element size; C
 * must not overlap A or B). Checks: lda >= K, ldb >= N, ldc >= N, all >= 1,
 * 0 <= stride_b < 2^40 (AC_ERR_INVALID_VALUE); lda or ldb >= AC_MAX_LD
 * (AC_ERR_UNSUPPORTED); a plan of adaptcore_plan given here, or a grouped
 * plan given to adaptcore_matmul: AC_ERR_INVALID_VALUE. rows, groups or N
 * equal to 0: nothing is launched. K == 0: the covered rows of C are set to
 * zero. The caller guarantees that B holds every group's matrix:
 * (groups - 1) * stride_b + (K - 1) * ldb + N elements. No workspace. */
adaptcore_status adaptcore_grouped_matmul(const adaptcore_plan_t* plan, const int32_t* counts, const void* A,
                                          int64_t lda, const void* B, int64_t ldb, int64_t stride_b, void* C,
                                          int64_t ldc, void* stream);

/* The grouped product with the AddMM epilogue of adaptcore_addmm (GroupMM
 * and AddMM, Section 6.5): the covered rows r of group g get
 * C[r] = alpha * (A[r] * B_g) + beta * C_old[r] + bias_g, in fp32 before the
 * rounding to C's type, C_old read only when beta != 0; bias_g is the row of
 * N fp32 values at bias + g * stride_bias (stride_bias = 0 shares one row;
 * bias NULL: none). Arguments and validation as adaptcore_grouped_matmul,
 * plus finite alpha and beta, a 4-byte-aligned bias and 0 <= stride_bias <
 * 2^40 (AC_ERR_INVALID_VALUE); the caller guarantees that bias holds
 * (groups - 1) * stride_bias + N values. Rows no group covers keep their
 * contents. */
adaptcore_status adaptcore_grouped_addmm(const adaptcore_plan_t* plan, const int32_t* counts, const void* A,
                                         int64_t lda, const void* B, int64_t ldb, int64_t stride_b, void* C,
                                         int64_t ldc, float alpha, float beta, const float* bias, int64_t stride_bias,
                                         void* stream);

/* ---- Batched product (BatchMM) ---------------------------------------------
 * The other batched operator the paper replaces in its end-to-end models
 * (BatchMM, Section 6.5; operator scope, Section 7), in the strided form:
 * for b = 0 .. batch-1,
 *     C_b = A_b * B_b,  A_b = A + b*stride_a (M x K, lda),
 *                        B_b = B + b*stride_b (K x N, ldb),
 *                        C_b = C + b*stride_c (M x N, ldc),
 * strides in elements (0 repeats one matrix for every batch). It runs on the
 * grouped product's kernel with every group the same shape: one launch, no
 * workspace, no device counts.
 *
 * Returns the cached plan for (batch, M, N, K, dtype, layouts): M, N, K in
 * [0, 2^31), batch in [0, 2^24]. NULL on invalid or unsupported arguments. */
const adaptcore_plan_t* adaptcore_batched_plan(int64_t batch, int64_t M, int64_t N, int64_t K, int32_t dtype,
                                               uint32_t layouts);

/* Like adaptcore_batched_plan with the configuration forced to variant_key
 * (family AC_FAMILY_BATCHED, P_k = 1). For tests. NULL if not legal. */
const adaptcore_plan_t* adaptcore_batched_plan_variant(int64_t batch, int64_t M, int64_t N, int64_t K,
                                                       int32_t dtype, uint32_t layouts, uint64_t variant_key);

/* Runs a batched plan asynchronously on `stream`. A, B, C device pointers
 * (A, B 2-byte aligned, C aligned to its element size; C must not overlap A
 * or B). Checks: lda >= K, ldb >= N, ldc >= N, all >= 1; strides in
 * [0, 2^40); for batch > 1, stride_c >= (M-1)*ldc + N so that no two C
 * matrices overlap (AC_ERR_INVALID_VALUE); lda or ldb >= AC_MAX_LD
 * (AC_ERR_UNSUPPORTED); a plan of another kind: AC_ERR_INVALID_VALUE.
 * batch, M or N equal to 0: nothing is launched. K == 0: C is set to zero.
 * The caller guarantees that A, B and C hold every batch's matrix. */
adaptcore_status adaptcore_batched_matmul(const adaptcore_plan_t* plan, const void* A, int64_t lda, int64_t stride_a,
                                          const void* B, int64_t ldb, int64_t stride_b, void* C, int64_t ldc,
                                          int64_t stride_c, void* stream);

/* The batched product with the AddMM epilogue of adaptcore_addmm (the
 * epilogues the paper's BatchMM and AddMM operators need, Section 6.5): for
 * every batch b, C_b = alpha * A_b * B_b + beta * C_b,old + bias, in fp32
 * before the rounding to C's type, C_b,old read only when beta != 0, bias a
 * device array of N fp32 values shared by all batches (NULL: none).
 * Arguments and validation as adaptcore_batched_matmul, plus finite alpha
 * and beta and a 4-byte-aligned bias (AC_ERR_INVALID_VALUE). K == 0 yields
 * C_b = beta * C_b,old + bias. */
adaptcore_status adaptcore_batched_addmm(const adaptcore_plan_t* plan, const void* A, int64_t lda, int64_t stride_a,
                                         const void* B, int64_t ldb, int64_t stride_b, void* C, int64_t ldc,
                                         int64_t stride_c, float alpha, float beta, const float* bias, void* stream);

/* Allocates (if needed) the workspace of `stream` for plans needing up to
 * `bytes`, so that later calls, also under capture, do not allocate. A
 * workspace that grows keeps its previous buffer alive (see
 * adaptcore_matmul). */
adaptcore_status adaptcore_reserve_workspace(void* stream, int64_t bytes);

/* Fills *out with the description of a plan: the template of the taxonomy
 * (Section 4.2), the selected configuration x* (Eq. 6) as its VariantKey,
 * the tiling (m1, n1, k1) and task counts P_m, P_n, P_k of Table 1, the
 * launch grid, the latency the model of Eqs. 7-14 predicts and the workspace
 * size. AC_ERR_INVALID_VALUE for a null argument. */
adaptcore_status adaptcore_plan_info(const adaptcore_plan_t* plan, adaptcore_plan_desc_t* out);

/* Writes the kernels one call of the plan launches, in launch order, as
 * "name<template arguments>" separated by ';' (the names a profiler shows,
 * without namespace and parameter list) into buf (capacity len bytes,
 * NUL-terminated). AC_ERR_INVALID_VALUE if buf is too small. */
adaptcore_status adaptcore_plan_kernels(const adaptcore_plan_t* plan, char* buf, int64_t len);

/* Lists the legal candidates of a shape with their model latencies, ordered
 * by the model's preference (best first). Returns the number of candidates
 * (which may exceed cap; at most cap are written), or a negative status. */
int64_t adaptcore_candidates(int64_t M, int64_t N, int64_t K, int32_t dtype, uint32_t layouts,
                             adaptcore_candidate_t* out, int64_t cap);

/* Planner profile. set() drops every cached plan (they depend on it) by
 * calling adaptcore_cache_clear: plans returned earlier become invalid, so
 * call it only when no other thread uses the library. */
adaptcore_status adaptcore_get_hw(adaptcore_hw_t* out);
adaptcore_status adaptcore_set_hw(const adaptcore_hw_t* hw);

adaptcore_status adaptcore_stats(adaptcore_stats_t* out);

/* Drops every cached plan. Plans returned earlier become invalid: call only
 * when no other thread uses the library. */
adaptcore_status adaptcore_cache_clear(void);

/* Median host time of one cached lookup, in nanoseconds, measured over
 * n_lookups lookups cycling through n_keys distinct shapes already planned
 * (timed in C, without any binding overhead). */
adaptcore_status adaptcore_bench_lookup(int64_t n_keys, int64_t n_lookups, double* ns_per_lookup);

/* Measurement reference, not part of the method: reads every byte of the
 * device buffer `buf` once (16-byte non-temporal loads, 8 in flight per
 * thread, two workgroups per CU) on `stream`, so that the time of a call is
 * the achievable HBM read rate for that many bytes -- the practical ceiling
 * of the kernels that stream one operand (the small-M / decode and
 * tall-skinny paths). `buf` 16-byte aligned, `bytes` a multiple of 16 (else
 * AC_ERR_INVALID_VALUE); `sink` a 4-byte aligned device word that is written
 * only if the XOR of all the data equals 0x9E3779B9. AC_ERR_LAUNCH if the
 * runtime rejects the launch. */
adaptcore_status adaptcore_read_probe(const void* buf, int64_t bytes, void* sink, void* stream);

/* Thread-local message of the last failure ("" if none). */
const char* adaptcore_last_error(void);

/* Thread-local status of the last failure (AC_OK if none), e.g. the reason an
 * adaptcore_plan call returned NULL. */
adaptcore_status adaptcore_last_status(void);

/* ---- planner arithmetic, exposed for testing against the paper ---------- */

/* The taxonomy and data-volume terms for explicit tiling parameters and a
 * hardware (n_core, s_acc): task counts (Table 1), the template of
 * Section 4.2, D_r of Eq. 1 and D_w of Eqs. 2-5 (bytes; elem_bytes and
 * out_bytes as Section 4.2 assumes fp16, i.e. 2 and 2). */
typedef struct {
  int64_t M, N, K, m, n, k, m1, n1, k1;
  int64_t n_core, s_acc;
  int32_t elem_bytes, out_bytes;
} adaptcore_taxonomy_in_t;
typedef struct {
  int64_t pm, pn, pk;
  int32_t cls;
  int64_t acc_bytes;
  double read_bytes;  /* Eq. 1 */
  double write_bytes; /* Eqs. 2-5 for the template */
} adaptcore_taxonomy_out_t;
adaptcore_status adaptcore_taxonomy(const adaptcore_taxonomy_in_t* in, adaptcore_taxonomy_out_t* out);

/* Pipeline schedules of Section 5.3: kind 0 = baseline (Eq. 12), 1 = double
 * buffering (Eq. 13), 2 = preloading over Q tiles (Eq. 14). */
double adaptcore_schedule(int32_t kind, int64_t Q, int64_t L, double t_m, double t_p, double t_drain);

#ifdef __cplusplus
}
#endif
#endif /* ADAPTCORE_H */
