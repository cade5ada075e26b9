// Launch registry: plan -> kernel on a stream.
#pragma once
#include <hip/hip_runtime_api.h>

#include "kernel_args.h"
#include "planner.h"

namespace ac {
// bf16 inputs (dtypes 0 and 1)
hipError_t launch_plan(const Plan& p, const GemmArgs& g, hipStream_t st);
// Direct-to-LDS tile kernels (kernels_dl.hip): whether the operands meet
// their alignment (16-byte aligned rows of A and B, K and N multiples of 8,
// lda and ldb below DL_MAX_LD; the same for both input formats), and the
// main kernel of a FAM_DL plan (the split-K reduction is launched by
// launch_plan).
bool dl_operands_aligned(const GemmArgs& g);
// The same test per operand (A: 16-byte aligned rows of K, K a multiple of
// 8; B: 16-byte aligned rows, nB a multiple of 8; lda, ldb below DL_MAX_LD).
bool dl_a_aligned(const void* A, int64_t lda, int64_t K);
bool dl_b_aligned(const void* B, int64_t ldb, int64_t nB);
// Padding prologue: dst (rows x ld_dst, ld_dst a multiple of 8 >= cols, dst
// 16-byte aligned) = src (rows x cols, row pitch ld_src) with zeros in the
// pad columns.
hipError_t launch_pad16(const uint16_t* src, int64_t ld_src, int64_t rows, int64_t cols, uint16_t* dst,
                        int64_t ld_dst, hipStream_t st);
hipError_t launch_dl_main(const Plan& p, const GemmArgs& g, hipStream_t st);
hipError_t launch_dl_sc_main(const Plan& p, const GemmArgs& g, hipStream_t st);
void query_occupancy_dl();
// Tall-skinny streaming kernel (kernels_tall.hip): A's alignment (16-byte
// aligned rows of K, K a multiple of 8, lda below DL_MAX_LD), the operands'
// (A and the transposed copy of B in g.B / g.ldb), and the main kernel of a
// FAM_TALL plan (the B^T prologue and the split-K reduction are launched by
// the caller and launch_plan).
bool tall_a_aligned(const void* A, int64_t lda, int64_t K);
bool tall_operands_aligned(const GemmArgs& g);
hipError_t launch_tall_main(const Plan& p, const GemmArgs& g, hipStream_t st);
void query_occupancy_tall();
// Launch of a grouped or batched plan (families FAM_GROUPED, FAM_BATCHED).
hipError_t launch_grouped_plan(const Plan& p, const GroupArgs& a, hipStream_t st);
// Reads the device's occupancy of every kernel into the planner.
void query_occupancy();
// Layout prologue: dst (cols x rows, row pitch ld_dst, a multiple of 8, dst
// 16-byte aligned) = transpose of the 16-bit matrix src (rows x cols, row
// pitch ld_src >= cols); the pad of each dst row is written with zeros.
hipError_t launch_transpose16(const uint16_t* src, int64_t ld_src, int64_t rows, int64_t cols, uint16_t* dst,
                              int64_t ld_dst, hipStream_t st);
// Measurement reference (not part of the product): reads every byte of
// `buf` once (16-byte aligned, `bytes` a multiple of 16).
hipError_t launch_read_probe(const void* buf, int64_t bytes, void* sink, hipStream_t st);
// the same kernels for fp16 inputs (dtypes 2 and 3)
namespace f16 {
hipError_t launch_plan(const Plan& p, const GemmArgs& g, hipStream_t st);
hipError_t launch_dl_main(const Plan& p, const GemmArgs& g, hipStream_t st);
hipError_t launch_dl_sc_main(const Plan& p, const GemmArgs& g, hipStream_t st);
void query_occupancy_dl();
hipError_t launch_tall_main(const Plan& p, const GemmArgs& g, hipStream_t st);
void query_occupancy_tall();
hipError_t launch_grouped_plan(const Plan& p, const GroupArgs& a, hipStream_t st);
void query_occupancy();
}  // namespace f16
}  // namespace ac
