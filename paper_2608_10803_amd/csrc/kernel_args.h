// Launch arguments shared by the host dispatcher and the gfx950 kernels.
#pragma once
#include <stdint.h>

namespace ac {

// Element types of adaptcore_dtype: 0 bf16 in / fp32 out, 1 bf16 in / bf16
// out, 2 fp16 in / fp32 out, 3 fp16 in / fp16 out.
constexpr bool dtype_f16_input(int dtype) { return dtype == 2 || dtype == 3; }
constexpr bool dtype_out16(int dtype) { return dtype == 1 || dtype == 3; }
constexpr int dtype_out_bytes(int dtype) { return dtype_out16(dtype) ? 2 : 4; }

// Kernel families of the variant space.
enum Family : int {
  FAM_TILE = 0,      // MFMA macro-tile kernel; P_k == 1 is the Common template,
                     // P_k > 1 the MultiCoreSplitK template (Section 4.2)
  FAM_SKINNY_M = 1,  // Small-M Copy module: B streamed once, M <= 64
  FAM_SKINNY_N = 2,  // the same module by orientation: A streamed once, N <= 64
  FAM_STREAMK = 3,   // StreamK applied to the tile kernel (Section 4.2)
  FAM_SMALLK = 4,    // K <= 16: rank-K update, bound by writing C
  FAM_DIRECT = 5,    // small problems: MFMA fragments loaded straight from memory
  FAM_GROUPED = 6,   // the tile kernel over the groups of a grouped product
  FAM_PERSIST = 7,   // persistent tile kernel, next tile's first block fetched before the epilogue
  FAM_BATCHED = 8,   // the grouped kernel over a strided batch (every group the same shape)
  FAM_DL = 9,        // tile kernel with operand tiles loaded straight into LDS (multi-stage)
  FAM_TALL = 10,     // N <= 32: A streamed once through a direct-to-LDS pipeline, B^T beside it
  FAM_DLSC = 11,     // off-chip accumulation: a workgroup's 2-tile super-tile, partials flushed per k1 slice
  FAM_COUNT = 12
};

// Arguments of every GEMM kernel. A is M x K row-major (lda), B is K x N
// row-major (ldb), C is M x N row-major (ldc); 16-bit inputs as raw bits.
struct GemmArgs {
  const uint16_t* A;
  const uint16_t* B;
  void* C;
  int64_t M, N, K;
  int64_t lda, ldb, ldc;
  float* ws;         // fp32 partials: split K uses pk slices of M x ldw,
                     // stream-K uses ws_pk row-major tiles per split tile
  int64_t ldw;       // leading dimension of a split-K partial slice (N rounded up to 8)
  int pk;            // K partitions (1 = no split)
  int kper;          // k-blocks per partition (block = the kernel's k granule)
  int tiles_m;       // output tiles along M of this kernel's tiling
  int tiles_n;       // output tiles along N
  int swizzle;       // 1 = XCD-aware, grouped tile order
  int iters_per_wg;  // stream-K: MAC iterations per persistent workgroup
  int sk_tiles;      // stream-K: tiles handled by the stream-K phase
  int ws_pk;         // stream-K: partial slots per split tile
  int grid;          // stream-K: persistent workgroups
  // AddMM epilogue (epi != 0): C = alpha * (A B) + beta * C_old + bias[col],
  // applied in fp32 where the final C is written; C_old is read only when
  // beta != 0. Partials of split K and stream-K stay raw sums.
  float alpha, beta;
  const float* bias;  // N values or null
  int epi;
  // Direct-to-LDS kernels: the rows of B (its real K) and the columns of B
  // that may be loaded (N, or N rounded up to 8 when B is a zero-padded
  // copy). K is then the k the loop runs over: rounded up to 8 when A is a
  // zero-padded copy. Other kernels ignore both.
  int64_t kB, nB;
};

// Arguments of the grouped kernel. With counts: group g owns rows
// [min(P_{g-1}, rows), min(P_g, rows)) of A and C (P: running sum of
// max(counts, 0)). Without counts (a strided batch): every group has `rows`
// rows, its A at A + g * stride_a and its C at C + g * stride_c. Either way
// group g multiplies its rows by the K x N matrix at B + g * stride_b. g.M is
// unused; g.tiles_n is the tile count along N.
struct GroupArgs {
  GemmArgs g;
  const int32_t* counts;  // device, `groups` entries; null = strided batch
  int64_t rows;           // rows of A and C (capacity), or rows of every batch
  int64_t stride_a;       // strided batch: elements between two A matrices (else 0)
  int64_t stride_b;       // elements between the B matrices of two groups
  int64_t stride_c;       // strided batch: elements between two C matrices (else 0)
  int64_t stride_bias;    // AddMM epilogue: fp32 values between the bias rows of two groups
  int groups;
  int slots;              // row-tile slots launched (an upper bound of the tiles along M)
  int tiles_per_group;    // strided batch: row tiles of every group
};

}  // namespace ac
