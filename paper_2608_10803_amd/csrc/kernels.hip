// gfx950 GEMM kernels: C = A * B with 16-bit inputs, fp32 accumulation and
// fp32 or 16-bit output (RNE), for any M, N, K, leading dimensions and 2-byte
// aligned pointers. The file is compiled twice: for bf16 inputs (namespace ac)
// and, with AC_INPUT_F16=1, for fp16 inputs (namespace ac::f16). Only the MFMA
// instructions, the 16-bit output rounding and the small-K kernel's input
// decode depend on the format; 16-bit outputs are in the input format.
//
//   k_tile      MFMA macro-tile kernel, LDS double buffered, one or two
//               k-blocks of global loads in flight. P_k == 1 is the Common template
//               (k = K, one cast and one write per output, Eq. 2); P_k > 1 the
//               MultiCoreSplitK template (each workgroup writes an fp32 partial
//               of its K range, Eq. 4; k_reduce then sums them, Eq. 11).
//   k_streamk   StreamK applied to the tile kernel (Section 4.2): a persistent
//               grid splits the MAC iterations of the last tiles evenly and
//               writes the pieces as fp32 partials; k_sk_fixup sums them.
//   k_skinny_m  Small-M Copy module (Table 2) for M <= 64: B is streamed from
//               HBM exactly once, A stays in cache; K split across CUs.
//   k_skinny_n  the same module for N <= 64: A streamed once, the small B is
//               kept resident in LDS (L1 Resident module, Table 2).
//   k_smallk    K <= 16: rank-K update with fp32 FMAs, bound by writing C once.
//   k_direct    small problems: MFMA fragments straight from global memory,
//               no LDS staging, the fewest instructions between load and store.
//   k_reduce    deterministic cross-workgroup reduction of split-K partials:
//               sum in partition order 0, 1, ..., P_k - 1, then cast.
//
// Workgroups never wait on each other: partials are combined by a second
// kernel, so a result never depends on arrival order and no kernel spins.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "kernel_args.h"
#include "variants.h"

#ifndef AC_INPUT_F16
#define AC_INPUT_F16 0
#endif

namespace ac {
#if AC_INPUT_F16
namespace f16 {
#endif

#include "device_common.h"

// ---------------------------------------------------------------- helpers

// Transpose an 8 x 8 block of 16-bit values: r[i] holds row i (8 columns),
// c[j] receives column j (8 rows), row 2e in the low half of dword e.
__device__ __forceinline__ void transpose8x8(const u32x4 (&r)[8], u32x4 (&c)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int d = j >> 1;
    const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
    for (int e = 0; e < 4; ++e) c[j][e] = __builtin_amdgcn_perm(r[2 * e + 1][d], r[2 * e][d], sel);
  }
}

// Eight consecutive outputs of one row; `valid` of them exist.
template <bool OBF>
__device__ __forceinline__ void store_c8(void* C, int64_t idx, const float (&v)[8], int64_t valid) {
  if constexpr (OBF) {
    uint16_t* p = static_cast<uint16_t*>(C) + idx;
    if (valid >= 8) {
      u32x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = (uint32_t)to16(v[2 * e]) | ((uint32_t)to16(v[2 * e + 1]) << 16);
      __builtin_memcpy(p, &w, 16);
    } else {
      for (int j = 0; j < valid; ++j) p[j] = to16(v[j]);
    }
  } else {
    float* p = static_cast<float*>(C) + idx;
    if (valid >= 8) {
      f32x4 w0 = {v[0], v[1], v[2], v[3]}, w1 = {v[4], v[5], v[6], v[7]};
      __builtin_memcpy(p, &w0, 16);
      __builtin_memcpy(p + 4, &w1, 16);
    } else {
      for (int j = 0; j < valid; ++j) p[j] = v[j];
    }
  }
}

// One / eight final outputs of C at (row, col): the epilogue, then the store.
template <bool OBF>
__device__ __forceinline__ void store_out(const GemmArgs& g, int64_t row, int64_t col, float v) {
  float w[1] = {v};
  epi_apply<OBF, 1>(g, w, row, col, 1);
  store_c<OBF>(g.C, row * g.ldc + col, w[0]);
}
template <bool OBF>
__device__ __forceinline__ void store_out8(const GemmArgs& g, int64_t row, int64_t col, const float (&v)[8],
                                           int64_t valid) {
  float w[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) w[e] = v[e];
  epi_apply<OBF, 8>(g, w, row, col, valid);
  store_c8<OBF>(g.C, row * g.ldc + col, w, valid);
}

// LDS rows are 16-byte chunks; the chunk index is XORed with low row bits so
// that the lanes reading consecutive rows at one chunk hit distinct banks.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row & 7) ^ ((row >> 3) & 1)); }

// ------------------------------------------------------------ tile kernel

template <int MS>
struct AccOf;
template <>
struct AccOf<32> {
  typedef f32x16 T;
  static constexpr int n = 16;
};
template <>
struct AccOf<16> {
  typedef f32x4 T;
  static constexpr int n = 4;
};

// Waves of a tile workgroup: 4 in a 2 x 2 grid, or 8 in a 2 x 4 grid for the
// 256-row tiles (two waves per SIMD hide each other's waits; measured faster
// than 4 waves for 256 x 256 and 256 x 128, slower for 128 x 256).
constexpr int tile_waves(int bm, int bn) { return bm == 256 ? 8 : 4; }

template <int BM, int BN, int MS>
struct TileShape {
  static constexpr int NW = tile_waves(BM, BN), WC = NW / 2;
  static constexpr int NT = 64 * NW, BK = 64, CH = 8;
  static constexpr int WTM = BM / 2, WTN = BN / WC;
  static constexpr int TM = WTM / MS, TN = WTN / MS;
  static constexpr int KS = MS == 32 ? 16 : 32;
  static constexpr int NA = AccOf<MS>::n;
  static constexpr int AV = BM * CH;  // 16-byte vectors of an A stage
  static constexpr int IA = (AV + NT - 1) / NT;
  // B stage: BK/8 * BN/8 = BN blocks of 8 k-rows x 8 columns; each block is
  // shared by BP threads, each taking BR = 8 / BP consecutive k-rows, so that
  // (where possible) every thread of the workgroup has one unit of B work.
  static constexpr int BP = (NT / BN >= 4) ? 4 : (NT / BN >= 2 ? 2 : 1);
  static constexpr int BR = 8 / BP;
  static constexpr int BU = BN * BP;                // B units of a stage
  static constexpr int IB = (BU + NT - 1) / NT;     // B units per thread
  static constexpr int AB_BYTES = 2 * (BM + BN) * CH * 16;  // double-buffered A and B stages
  static constexpr int CT_LD = BN + 4;                        // padded LDS row of the output tile
  static constexpr int CT_BYTES = BM * CT_LD * 2;             // bf16 output tile
  static constexpr int SMEM = AB_BYTES > CT_BYTES ? AB_BYTES : CT_BYTES;
  static_assert(WTM % MS == 0 && WTN % MS == 0, "wave tile must be a multiple of the MFMA tile");
};

// Per-thread load geometry of a tile's stages (fixed for the tile). Offsets
// are 32-bit byte offsets from the per-k-block uniform bases
// A + m0*lda + kbase and B + kbase*ldb + n0; rows past M are clamped to row
// M - 1 (their results are never stored). For B, the 16-byte column group of
// a lane starts at min(gn, N - 8), so it never leaves the row; the lanes that
// had to move left drop the extra leading elements when the stage goes to LDS.
template <int BM, int BN, int MS>
struct StageGeom {
  typedef TileShape<BM, BN, MS> S;
  uint32_t a_row[S::IA];  // bytes: clamped row * lda * 2 + 16
  uint32_t b_col[S::IB];  // bytes: (start column - n0) * 2 + 16 (>= 0: start >= n0 - 8)
  int32_t b_cs[S::IB];    // elements dropped at the N edge: 0..8 (8 = past N)
  uint32_t ldb2;          // bytes per B row
  __device__ __forceinline__ void init(const GemmArgs& g, int64_t m0, int64_t n0) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < S::IA; ++i) {
      const int row = (tid + i * S::NT) >> 3;
      a_row[i] = (uint32_t)((min(m0 + row, g.M - 1) - m0) * g.lda * 2 + 16);
    }
#pragma unroll
    for (int bb = 0; bb < S::IB; ++bb) {
      const int grp = (min(tid + bb * S::NT, S::BU - 1) / S::BP) >> 3;
      const int64_t gn = n0 + grp * 8;
      const int64_t st = min(gn, g.N - 8);
      b_col[bb] = (uint32_t)((st - n0) * 2 + 16);
      b_cs[bb] = (int32_t)min(gn - st, (int64_t)8);
    }
    ldb2 = (uint32_t)(g.ldb * 2);
  }
};

// base (uniform) + unsigned 32-bit byte offset: lets the compiler use the
// scalar-base + vector-offset addressing of global loads.
__device__ __forceinline__ const uint16_t* at(const uint16_t* base, uint32_t byte_off) {
  return reinterpret_cast<const uint16_t*>(reinterpret_cast<const char*>(base) + byte_off);
}

// Global loads of one k-block stage into registers, then into LDS. The loads
// are straight-line code for every block (interior or edge): a K tail moves
// the A vectors left to end at the row end and clamps the B rows, exactly as
// the N edge does for B columns; the recorded shifts are applied when the
// stage is written to LDS, after all loads of the stage have been issued.
template <int BM, int BN, int MS>
struct Stage {
  typedef TileShape<BM, BN, MS> S;
  u32x4 ra[S::IA];
  u32x4 rb[S::IB][S::BR];
  uint32_t code;  // bits 0-3: A elements to drop; bits 4-11: B rows past K

  // Requires K >= 8 and N >= 8 (the small-row mode covers the rest). A
  // thread's A vectors all sit at column (tid % 8) * 8 of the block and its B
  // blocks all start at k-row (tid % 8) * 8, so one shift and one row mask
  // serve all of them.
  __device__ __forceinline__ void load(const GemmArgs& g, const StageGeom<BM, BN, MS>& o, int64_t m0,
                                       int64_t n0, int kt) {
    const int tid = threadIdx.x;
    const int64_t kbase = (int64_t)kt * S::BK;
    const int rem = (int)min(g.K - kbase, (int64_t)(1 << 30));  // K left from this block on (uniform)
    // bases 8 elements left of the block origin: every offset is >= 0
    const uint16_t* Ab = g.A + m0 * g.lda + kbase - 8;
    const uint16_t* Bb = g.B + kbase * g.ldb + n0 - 8;
    const int c8 = (tid & 7) * 8;
    const int st = min(c8, rem - 8);  // >= -8
    uint32_t cd = (uint32_t)min(c8 - st, 8);
#pragma unroll
    for (int i = 0; i < S::IA; ++i)
      if (S::AV % S::NT == 0 || tid + i * S::NT < S::AV) ra[i] = load16(at(Ab, o.a_row[i] + (uint32_t)(st * 2)));
    // B: this thread's rows of its block(s): k-rows (blk % 8) * 8 + part * BR
    // + i, where unit u = tid + b * NT = blk * BP + part; all units of a
    // thread share blk % 8 and part (NT is a multiple of 8 * BP)
    const int bk0 = ((tid / S::BP) & 7) * 8 + (tid % S::BP) * S::BR;
#pragma unroll
    for (int i = 0; i < S::BR; ++i) {
      const int kr = min(bk0 + i, rem - 1);
      cd |= (uint32_t)(bk0 + i >= rem) << (4 + i);
#pragma unroll
      for (int b = 0; b < S::IB; ++b)
        if (S::BU % S::NT == 0 || tid + b * S::NT < S::BU)  // uniform over a wave
          rb[b][i] = load16(at(Bb, (uint32_t)kr * o.ldb2 + o.b_col[b]));
    }
    code = cd;
  }

  // Small-row mode (K < 8 or N < 8): element loads, zeros outside the matrix.
  __device__ __forceinline__ void load_small(const GemmArgs& g, int64_t m0, int64_t n0, int kt) {
    const int tid = threadIdx.x;
    const int64_t kbase = (int64_t)kt * S::BK;
    code = 0;
#pragma unroll
    for (int i = 0; i < S::IA; ++i) {
      const int idx = tid + i * S::NT;
      if (S::AV % S::NT == 0 || idx < S::AV) {
        const int64_t gr = min(m0 + (idx >> 3), g.M - 1), gk = kbase + (idx & 7) * 8;
        ra[i] = load_row8_small(g.A + gr * g.lda, gk, g.K);
        __builtin_amdgcn_sched_barrier(0);  // one vector at a time: few live registers
      }
    }
#pragma unroll
    for (int b = 0; b < S::IB; ++b) {
      const int u = tid + b * S::NT;
      if (S::BU % S::NT == 0 || u < S::BU) {
        const int blk = u / S::BP, part = u % S::BP;
        const int64_t gn = n0 + (blk >> 3) * 8;
#pragma unroll
        for (int i = 0; i < S::BR; ++i) {
          const int64_t gk = kbase + (blk & 7) * 8 + part * S::BR + i;
          const u32x4 v = load_row8_small(g.B + min(gk, g.K - 1) * g.ldb, gn, g.N);
          rb[b][i] = gk < g.K ? v : u32x4{0u, 0u, 0u, 0u};
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  }

  // edge: this stage's block needed shifts (uniform flag); `cs` is the
  // tile's B column shift of this thread's blocks (StageGeom::b_cs).
  __device__ __forceinline__ void store(u32x4* sA, u32x4* sB, bool edge, const int32_t (&cs)[S::IB]) {
    const int tid = threadIdx.x;
    if (edge) {
      const int sa = (int)(code & 15);
#pragma unroll
      for (int i = 0; i < S::IA; ++i) ra[i] = shift_down(ra[i], sa);
#pragma unroll
      for (int b = 0; b < S::IB; ++b)
#pragma unroll
        for (int i = 0; i < S::BR; ++i) rb[b][i] = shift_down(rb[b][i], ((code >> (4 + i)) & 1) ? 8 : cs[b]);
    }
#pragma unroll
    for (int i = 0; i < S::IA; ++i) {
      const int idx = tid + i * S::NT;
      if (S::AV % S::NT == 0 || idx < S::AV) {
        const int row = idx >> 3, c = idx & 7;
        sA[row * 8 + swz(row, c)] = ra[i];
      }
    }
#pragma unroll
    for (int b = 0; b < S::IB; ++b) {
      const int u = tid + b * S::NT;
      if (S::BU % S::NT == 0 || u < S::BU) {
        const int blk = u / S::BP, part = u % S::BP;
        const int c = blk & 7, grp = blk >> 3;
        if constexpr (S::BR == 8) {
          u32x4 col[8];
          transpose8x8(rb[b], col);
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int n = grp * 8 + j;
            sB[n * 8 + swz(n, c)] = col[j];
          }
        } else {
          // column j of this thread's BR rows: BR / 2 dwords, written into
          // part `part` of the column's 16-byte k-chunk
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int n = grp * 8 + j, d = j >> 1;
            const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
            uint32_t* dst = reinterpret_cast<uint32_t*>(&sB[n * 8 + swz(n, c)]) + part * (S::BR / 2);
            if constexpr (S::BR == 4) {
              const uint32_t w0 = __builtin_amdgcn_perm(rb[b][1][d], rb[b][0][d], sel);
              const uint32_t w1 = __builtin_amdgcn_perm(rb[b][3][d], rb[b][2][d], sel);
              const uint64_t w = (uint64_t)w0 | ((uint64_t)w1 << 32);
              *reinterpret_cast<uint64_t*>(dst) = w;
            } else {
              *dst = __builtin_amdgcn_perm(rb[b][1][d], rb[b][0][d], sel);
            }
          }
        }
      }
    }
  }
};

// k-blocks of global loads in flight of the stream-K kernel (the tile kernel
// takes it from its configuration): two where the registers allow it.
constexpr int streamk_depth(int bm, int bn) { return (bm * bn <= 64 * 64 || (bm == 128 && bn == 256)) ? 2 : 1; }

// Accumulates the tile over k-blocks [kt0, kt1). With two stages in flight,
// block kt is multiplied out of LDS while block kt+1 waits in registers and
// block kt+2 is fetched. SMALL selects the element-load mode for K < 8 or
// N < 8 (decided once per kernel, so the loop body has no per-block branches).
template <int BM, int BN, int MS, int DEPTH, bool SMALL>
__device__ __forceinline__ void tile_mainloop_impl(const GemmArgs& g, int64_t m0, int64_t n0, int kt0, int kt1,
                                                   typename AccOf<MS>::T (&acc)[TileShape<BM, BN, MS>::TM]
                                                                              [TileShape<BM, BN, MS>::TN],
                                                   char* smem) {
  typedef TileShape<BM, BN, MS> S;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wr = wave / S::WC, wc = wave % S::WC;
  u32x4* sA0 = reinterpret_cast<u32x4*>(smem);
  u32x4* sA1 = sA0 + BM * 8;
  u32x4* sB0 = sA1 + BM * 8;
  u32x4* sB1 = sB0 + BN * 8;

  const int kt_total = (int)((g.K + S::BK - 1) / S::BK);
  const bool k_tail = (g.K % S::BK) != 0;
  const bool n_edge = n0 + BN > g.N;
  auto edge = [&](int kt) { return !SMALL && (n_edge || (k_tail && kt == kt_total - 1)); };

  auto compute = [&](const u32x4* sA, const u32x4* sB) {
#pragma unroll
    for (int ks = 0; ks < S::BK / S::KS; ++ks) {
      const int chunk = MS == 32 ? ks * 2 + (lane >> 5) : ks * 4 + (lane >> 4);
      u32x4 fa[S::TM], fb[S::TN];
#pragma unroll
      for (int i = 0; i < S::TM; ++i) {
        const int row = wr * S::WTM + i * MS + (lane % MS);
        fa[i] = sA[row * 8 + swz(row, chunk)];
      }
#pragma unroll
      for (int j = 0; j < S::TN; ++j) {
        const int col = wc * S::WTN + j * MS + (lane % MS);
        fb[j] = sB[col * 8 + swz(col, chunk)];
      }
#pragma unroll
      for (int i = 0; i < S::TM; ++i)
#pragma unroll
        for (int j = 0; j < S::TN; ++j) {
          // operands swapped: the MFMA forms the transposed tile, so a lane
          // holds one row of C and runs of 4 consecutive columns
          if constexpr (MS == 32)
            acc[i][j] = mfma32(fb[j], fa[i], acc[i][j]);
          else
            acc[i][j] = mfma16(fb[j], fa[i], acc[i][j]);
        }
    }
  };

  StageGeom<BM, BN, MS> o;
  o.init(g, m0, n0);  // (unused in the small-row mode)
  auto load = [&](Stage<BM, BN, MS>& st, int kt) {
    if constexpr (SMALL)
      st.load_small(g, m0, n0, kt);
    else
      st.load(g, o, m0, n0, kt);
  };

  // The loop bodies are straight-line (no per-lane branch, so no conservative
  // wait at a branch join splits the pipeline) and every load they issue is
  // of a block that is used: the last blocks are peeled off the loops.
  if constexpr (DEPTH == 1) {
    Stage<BM, BN, MS> st;
    load(st, kt0);
    st.store(sA0, sB0, edge(kt0), o.b_cs);
    __syncthreads();
    int kt = kt0;
    for (; kt + 1 < kt1; ++kt) {
      const bool odd = ((kt - kt0) & 1) != 0;  // uniform
      load(st, kt + 1);
      compute(odd ? sA1 : sA0, odd ? sB1 : sB0);
      st.store(odd ? sA0 : sA1, odd ? sB0 : sB1, edge(kt + 1), o.b_cs);
      __syncthreads();
    }
    const bool odd = ((kt - kt0) & 1) != 0;
    compute(odd ? sA1 : sA0, odd ? sB1 : sB0);
  } else {
    Stage<BM, BN, MS> s0, s1;
    if (kt0 + 1 == kt1) {  // a single block
      load(s0, kt0);
      s0.store(sA0, sB0, edge(kt0), o.b_cs);
      __syncthreads();
      compute(sA0, sB0);
      return;
    }
    load(s0, kt0);
    load(s1, kt0 + 1);
    s0.store(sA0, sB0, edge(kt0), o.b_cs);
    __syncthreads();
    int kt = kt0;
    for (; kt + 3 < kt1; kt += 2) {  // blocks kt + 2 and kt + 3 exist
      load(s0, kt + 2);
      compute(sA0, sB0);
      s1.store(sA1, sB1, edge(kt + 1), o.b_cs);
      __syncthreads();
      load(s1, kt + 3);
      compute(sA1, sB1);
      s0.store(sA0, sB0, edge(kt + 2), o.b_cs);
      __syncthreads();
    }
    if (kt + 2 < kt1) {  // three blocks left: kt (in LDS), kt + 1 (in s1), kt + 2
      load(s0, kt + 2);
      compute(sA0, sB0);
      s1.store(sA1, sB1, edge(kt + 1), o.b_cs);
      __syncthreads();
      compute(sA1, sB1);
      s0.store(sA0, sB0, edge(kt + 2), o.b_cs);
      __syncthreads();
      compute(sA0, sB0);
    } else {  // two blocks left: kt (in LDS), kt + 1 (in s1)
      compute(sA0, sB0);
      s1.store(sA1, sB1, edge(kt + 1), o.b_cs);
      __syncthreads();
      compute(sA1, sB1);
    }
  }
}

template <int BM, int BN, int MS, int DEPTH>
__device__ __forceinline__ void tile_mainloop(const GemmArgs& g, int64_t m0, int64_t n0, int kt0, int kt1,
                                              typename AccOf<MS>::T (&acc)[TileShape<BM, BN, MS>::TM]
                                                                         [TileShape<BM, BN, MS>::TN],
                                              char* smem) {
  if (kt0 >= kt1) return;
  if (g.K < 8 || g.N < 8)
    tile_mainloop_impl<BM, BN, MS, DEPTH, true>(g, m0, n0, kt0, kt1, acc, smem);
  else
    tile_mainloop_impl<BM, BN, MS, DEPTH, false>(g, m0, n0, kt0, kt1, acc, smem);
}

// Column (within the MFMA block) of accumulator element r of this lane; the
// lane's row is lane % MS (the MFMA forms the transposed block). Elements
// 4q .. 4q+3 are four consecutive columns.
template <int MS>
__device__ __forceinline__ int acc_col(int r, int lane) {
  if constexpr (MS == 32)
    return (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
  else
    return (lane >> 4) * 4 + r;
}

// fp32 store of the accumulators to a row-major matrix (C or a partial),
// rows < rmax and columns < cmax only.
template <int BM, int BN, int MS>
__device__ __forceinline__ void store_acc_f32(const typename AccOf<MS>::T (&acc)[TileShape<BM, BN, MS>::TM]
                                                                            [TileShape<BM, BN, MS>::TN],
                                              float* dst, int64_t ld, int64_t m0, int64_t n0, int64_t rmax,
                                              int64_t cmax, const GemmArgs* ep = nullptr) {
  typedef TileShape<BM, BN, MS> S;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wr = wave / S::WC, wc = wave % S::WC;
#pragma unroll
  for (int i = 0; i < S::TM; ++i) {
    const int64_t row = m0 + wr * S::WTM + i * MS + (lane % MS);
    if (row >= rmax) continue;
#pragma unroll
    for (int j = 0; j < S::TN; ++j)
#pragma unroll
      for (int q = 0; q < S::NA / 4; ++q) {
        // elements 4q .. 4q+3: four consecutive columns of the lane's row
        const int64_t col = n0 + wc * S::WTN + j * MS + acc_col<MS>(4 * q, lane);
        float* d = dst + row * ld + col;
        float w[4] = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
        if (ep != nullptr && col < cmax) epi_apply<false, 4>(*ep, w, row, col, cmax - col);
        if (col + 4 <= cmax) {
          const f32x4 v = {w[0], w[1], w[2], w[3]};
          __builtin_memcpy(d, &v, 16);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (col + e < cmax) d[e] = w[e];
        }
      }
  }
}

// bf16 output through LDS: the tile is converted into LDS row-major (rows
// padded to BN + 4 elements), then written with 16-byte row segments.
template <int BM, int BN, int MS, bool EPI>
__device__ __forceinline__ void store_acc_bf16(const typename AccOf<MS>::T (&acc)[TileShape<BM, BN, MS>::TM]
                                                                             [TileShape<BM, BN, MS>::TN],
                                               const GemmArgs& g, int64_t m0, int64_t n0, char* smem) {
  typedef TileShape<BM, BN, MS> S;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave / S::WC, wc = wave % S::WC;
  uint16_t* ct = reinterpret_cast<uint16_t*>(smem);
  __syncthreads();  // the main loop's last reads of the LDS stages are done
  // the lane's row of each MFMA tile, written 4 columns (8 bytes) at a time
#pragma unroll
  for (int i = 0; i < S::TM; ++i)
#pragma unroll
    for (int j = 0; j < S::TN; ++j) {
      // rows padded by 8 bytes: the 32 lanes writing 32 rows of one column
      // group fall on different banks
      uint16_t* base = ct + (wr * S::WTM + i * MS + (lane % MS)) * S::CT_LD + wc * S::WTN + j * MS;
#pragma unroll
      for (int q = 0; q < S::NA / 4; ++q) {
        float w[4] = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
        if (EPI && g.epi) {
          const int64_t row = m0 + wr * S::WTM + i * MS + (lane % MS);
          const int64_t col = n0 + wc * S::WTN + j * MS + acc_col<MS>(4 * q, lane);
          if (row < g.M && col < g.N) epi_apply<true, 4>(g, w, row, col, g.N - col);
        }
        const uint32_t lo = (uint32_t)to16(w[0]) | ((uint32_t)to16(w[1]) << 16);
        const uint32_t hi = (uint32_t)to16(w[2]) | ((uint32_t)to16(w[3]) << 16);
        const uint64_t v = (uint64_t)lo | ((uint64_t)hi << 32);
        *reinterpret_cast<uint64_t*>(base + acc_col<MS>(4 * q, lane)) = v;
      }
      __builtin_amdgcn_sched_barrier(0);  // convert block by block (bounded live registers)
    }
  __syncthreads();
  constexpr int GPR = BN / 8;  // 16-byte groups per tile row
  uint16_t* C = static_cast<uint16_t*>(g.C);
  for (int e = tid; e < BM * GPR; e += S::NT) {
    const int row = e / GPR, grp = e % GPR;
    const int64_t gr = m0 + row, gc = n0 + grp * 8;
    if (gr >= g.M || gc >= g.N) continue;
    const uint16_t* src = ct + row * S::CT_LD + grp * 8;
    uint16_t* dst = C + gr * g.ldc + gc;
    if (gc + 8 <= g.N) {
      // the padded rows are 8-byte aligned in LDS: two 8-byte reads
      const uint64_t lo = *reinterpret_cast<const uint64_t*>(src);
      const uint64_t hi = *reinterpret_cast<const uint64_t*>(src + 4);
      const uint64_t v[2] = {lo, hi};
      __builtin_memcpy(dst, v, 16);
    } else {
      for (int j = 0; j < (int)(g.N - gc); ++j) dst[j] = src[j];
    }
  }
}

template <int BM, int BN, int MS, bool OBF, bool EPI = false>
__device__ __forceinline__ void store_tile_c(const typename AccOf<MS>::T (&acc)[TileShape<BM, BN, MS>::TM]
                                                                           [TileShape<BM, BN, MS>::TN],
                                             const GemmArgs& g, int64_t m0, int64_t n0, char* smem) {
  if constexpr (OBF)
    store_acc_bf16<BM, BN, MS, EPI>(acc, g, m0, n0, smem);
  else
    store_acc_f32<BM, BN, MS>(acc, static_cast<float*>(g.C), g.ldc, m0, n0, g.M, g.N, EPI ? &g : nullptr);
}

// Output of the tile kernel: C in fp32, C in bf16, or (P_k > 1) the fp32
// partial of the workgroup's K partition.
enum TileOut : int { OUT_F32 = 0, OUT_BF16 = 1, OUT_PARTIAL = 2 };

template <int BM, int BN, int MS, int OUT, int DEPTH, bool EPI>
__device__ __forceinline__ void tile_kernel(const GemmArgs& g) {
  typedef TileShape<BM, BN, MS> S;
  typedef typename AccOf<MS>::T Acc;
  __shared__ __attribute__((aligned(16))) char smem[S::SMEM];

  const int ntiles = g.tiles_m * g.tiles_n;
  int tile = blockIdx.x;
  if (g.swizzle) tile = xcd_remap(tile, ntiles);
  int tm, tn;
  tile_coords(tile, g.tiles_m, g.tiles_n, g.swizzle, tm, tn);
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const int split = blockIdx.y;
  const int kt_total = (int)((g.K + S::BK - 1) / S::BK);
  const int kt0 = min(split * g.kper, kt_total);
  const int kt1 = min(kt0 + g.kper, kt_total);

  Acc acc[S::TM][S::TN];
#pragma unroll
  for (int i = 0; i < S::TM; ++i)
#pragma unroll
    for (int j = 0; j < S::TN; ++j) acc[i][j] = Acc{};

  tile_mainloop<BM, BN, MS, DEPTH>(g, m0, n0, kt0, kt1, acc, smem);

  if constexpr (OUT == OUT_PARTIAL)  // this partition's fp32 partial, row-major slice `split`
    store_acc_f32<BM, BN, MS>(acc, g.ws + (size_t)split * (size_t)g.M * (size_t)g.ldw, g.ldw, m0, n0, g.M, g.N);
  else
    store_tile_c<BM, BN, MS, OUT == OUT_BF16, EPI>(acc, g, m0, n0, smem);
}

// The tile kernel, and its form with the AddMM epilogue (a kernel of its own,
// so that the epilogue's registers never weigh on the plain product).
template <int BM, int BN, int MS, int OUT, int DEPTH>
__global__ __launch_bounds__(64 * tile_waves(BM, BN)) void k_tile(GemmArgs g) {
  tile_kernel<BM, BN, MS, OUT, DEPTH, false>(g);
}
template <int BM, int BN, int MS, int OUT, int DEPTH>
__global__ __launch_bounds__(64 * tile_waves(BM, BN)) void k_tile_addmm(GemmArgs g) {
  tile_kernel<BM, BN, MS, OUT, DEPTH, true>(g);
}

// ------------------------------------------------- persistent tile kernel
// Epilogues of the persistent kernel. Every thread issues the same, fixed
// number of 16-byte stores through a buffer resource whose range ends at the
// tile's last element of C; a lane whose 16 bytes lie outside C stores at an
// offset past that range, which the hardware drops. With a fixed count the
// compiler knows how many stores follow the next tile's prefetched loads, so
// waiting for those loads does not wait for the stores (vector memory
// operations complete in issue order). Only a last, partial group of columns
// (N not a multiple of 8) adds element stores. Requires the tile's span of C
// below 2^31 bytes (the launcher checks ldc). bf16 output only; fp32 output
// keeps the conditional register-to-memory stores.

template <int BM, int BN, int MS, bool EPI>
__device__ __forceinline__ void store_acc_bf16_fixed(const typename AccOf<MS>::T (&acc)[TileShape<BM, BN, MS>::TM]
                                                                                   [TileShape<BM, BN, MS>::TN],
                                                     const GemmArgs& g, int64_t m0, int64_t n0, char* smem) {
  typedef TileShape<BM, BN, MS> S;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave / S::WC, wc = wave % S::WC;
  uint16_t* ct = reinterpret_cast<uint16_t*>(smem);
  __syncthreads();  // the main loop's last reads of the LDS stages are done
#pragma unroll
  for (int i = 0; i < S::TM; ++i)
#pragma unroll
    for (int j = 0; j < S::TN; ++j) {
      uint16_t* base = ct + (wr * S::WTM + i * MS + (lane % MS)) * S::CT_LD + wc * S::WTN + j * MS;
#pragma unroll
      for (int q = 0; q < S::NA / 4; ++q) {
        float w[4] = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
        if (EPI && g.epi) {
          const int64_t row = m0 + wr * S::WTM + i * MS + (lane % MS);
          const int64_t col = n0 + wc * S::WTN + j * MS + acc_col<MS>(4 * q, lane);
          if (row < g.M && col < g.N) epi_apply<true, 4>(g, w, row, col, g.N - col);
        }
        const uint32_t lo = (uint32_t)to16(w[0]) | ((uint32_t)to16(w[1]) << 16);
        const uint32_t hi = (uint32_t)to16(w[2]) | ((uint32_t)to16(w[3]) << 16);
        *reinterpret_cast<uint64_t*>(base + acc_col<MS>(4 * q, lane)) = (uint64_t)lo | ((uint64_t)hi << 32);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  __syncthreads();
  constexpr int GPR = BN / 8;  // 16-byte groups per tile row
  constexpr int ITER = BM * GPR / S::NT;
  static_assert(BM * GPR % S::NT == 0, "whole store rounds");
  const int rows = (int)min(g.M - m0, (int64_t)BM), cols = (int)min(g.N - n0, (int64_t)BN);
  // the row pitch is made opaque here so that the per-store offsets are
  // computed in the epilogue, not hoisted out of the tile loop (where they
  // would stay live through the main loop)
  int32_t ldc2 = (int32_t)(g.ldc * 2);
  asm volatile("" : "+s"(ldc2));
  uint16_t* cbase = static_cast<uint16_t*>(g.C) + m0 * g.ldc + n0;
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(cbase, (short)0, (rows - 1) * ldc2 + cols * 2, (int)RSRC_WORD3);
  // in batches of at most 8 stores (bounded live registers)
  constexpr int BATCH = ITER < 8 ? ITER : 8;
  static_assert(ITER % BATCH == 0, "whole batches");
#pragma unroll
  for (int i0 = 0; i0 < ITER; i0 += BATCH) {
    u32x4 v[BATCH];
    int32_t off[BATCH];
#pragma unroll
    for (int u = 0; u < BATCH; ++u) {
      const int e = tid + (i0 + u) * S::NT, row = e / GPR, grp = e % GPR;
      const uint16_t* src = ct + row * S::CT_LD + grp * 8;  // 8-byte aligned
      const uint64_t a = *reinterpret_cast<const uint64_t*>(src);
      const uint64_t b = *reinterpret_cast<const uint64_t*>(src + 4);
      v[u] = u32x4{(uint32_t)a, (uint32_t)(a >> 32), (uint32_t)b, (uint32_t)(b >> 32)};
      const bool ok = row < rows && grp * 8 + 8 <= cols;
      off[u] = ok ? row * ldc2 + grp * 16 : OOB_OFF;
    }
#pragma unroll
    for (int u = 0; u < BATCH; ++u) __builtin_amdgcn_raw_buffer_store_b128(v[u], rs, off[u], 0, 0);
  }
  if ((cols & 7) != 0) {  // a partial last group of columns (uniform)
    const int c0 = cols & ~7;
    for (int r = tid; r < rows; r += S::NT)
      for (int j = c0; j < cols; ++j) cbase[(int64_t)r * g.ldc + j] = ct[r * S::CT_LD + j];
  }
}

// A grid of at most (CUs x workgroups per CU) walks the tiles in strides of
// the grid. The first k-block of a workgroup's next tile is loaded into
// registers right after the last k-block of the current tile went to LDS,
// i.e. before the current tile's last MFMAs and its epilogue, and goes to LDS
// at the end of the iteration: its memory latency is spent under the stores
// of C. Requires K >= 8 and N >= 8 (the planner offers it only then) and a
// row pitch of C below 2^23 bytes (the launcher checks it).
template <int BM, int BN, int MS, bool OBF, bool EPI>
__device__ __forceinline__ void persist_kernel(const GemmArgs& g) {
  typedef TileShape<BM, BN, MS> S;
  typedef typename AccOf<MS>::T Acc;
  __shared__ __attribute__((aligned(16))) char smem[S::SMEM];
  u32x4* sA0 = reinterpret_cast<u32x4*>(smem);
  u32x4* sA1 = sA0 + BM * 8;
  u32x4* sB0 = sA1 + BM * 8;
  u32x4* sB1 = sB0 + BN * 8;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wr = wave / S::WC, wc = wave % S::WC;

  const int ntiles = g.tiles_m * g.tiles_n;
  const int kt_total = (int)((g.K + S::BK - 1) / S::BK);
  const bool k_tail = (g.K % S::BK) != 0;
  int t = blockIdx.x;
  if (t >= ntiles) return;
  auto coords = [&](int tt, int64_t& m0, int64_t& n0) {
    const int tile = g.swizzle ? xcd_remap(tt, ntiles) : tt;
    int tm, tn;
    tile_coords(tile, g.tiles_m, g.tiles_n, g.swizzle, tm, tn);
    m0 = (int64_t)tm * BM;
    n0 = (int64_t)tn * BN;
  };
  auto compute = [&](const u32x4* sA, const u32x4* sB, Acc (&acc)[S::TM][S::TN]) {
#pragma unroll
    for (int ks = 0; ks < S::BK / S::KS; ++ks) {
      const int chunk = MS == 32 ? ks * 2 + (lane >> 5) : ks * 4 + (lane >> 4);
      u32x4 fa[S::TM], fb[S::TN];
#pragma unroll
      for (int i = 0; i < S::TM; ++i) {
        const int row = wr * S::WTM + i * MS + (lane % MS);
        fa[i] = sA[row * 8 + swz(row, chunk)];
      }
#pragma unroll
      for (int j = 0; j < S::TN; ++j) {
        const int col = wc * S::WTN + j * MS + (lane % MS);
        fb[j] = sB[col * 8 + swz(col, chunk)];
      }
#pragma unroll
      for (int i = 0; i < S::TM; ++i)
#pragma unroll
        for (int j = 0; j < S::TN; ++j) {
          if constexpr (MS == 32)
            acc[i][j] = mfma32(fb[j], fa[i], acc[i][j]);
          else
            acc[i][j] = mfma16(fb[j], fa[i], acc[i][j]);
        }
    }
  };

  int64_t m0, n0;
  coords(t, m0, n0);
  StageGeom<BM, BN, MS> o;
  o.init(g, m0, n0);
  Stage<BM, BN, MS> st;
  st.load(g, o, m0, n0, 0);
  bool n_edge = n0 + BN > g.N;
  st.store(sA0, sB0, n_edge || (k_tail && kt_total == 1), o.b_cs);
  __syncthreads();
  for (;;) {
    // block 0 of tile t is in LDS stage 0
    Acc acc[S::TM][S::TN];
#pragma unroll
    for (int i = 0; i < S::TM; ++i)
#pragma unroll
      for (int j = 0; j < S::TN; ++j) acc[i][j] = Acc{};
    int kt = 0;
    for (; kt + 1 < kt_total; ++kt) {
      const bool odd = (kt & 1) != 0;
      st.load(g, o, m0, n0, kt + 1);
      compute(odd ? sA1 : sA0, odd ? sB1 : sB0, acc);
      st.store(odd ? sA0 : sA1, odd ? sB0 : sB1, n_edge || (k_tail && kt + 1 == kt_total - 1), o.b_cs);
      __syncthreads();
    }
    // the last block of this tile is in LDS: fetch the next tile's first
    // block now, finish this tile, then move the block to LDS
    const int t_next = t + (int)gridDim.x;
    const bool more = t_next < ntiles;
    int64_t m1 = 0, n1 = 0;
    if (more) {
      coords(t_next, m1, n1);
      o.init(g, m1, n1);
      st.load(g, o, m1, n1, 0);
    }
    const bool odd = (kt & 1) != 0;
    compute(odd ? sA1 : sA0, odd ? sB1 : sB0, acc);
    // The fixed-count epilogue for bf16 output; fp32 output and the 256 x 256
    // tile keep the conditional stores (their fixed-count forms keep more
    // registers live than those tiles afford: spills, whose reloads wait for
    // every memory operation, cost more than the overlap gains).
    if constexpr (OBF && !(BM == 256 && BN == 256))
      store_acc_bf16_fixed<BM, BN, MS, EPI>(acc, g, m0, n0, smem);
    else
      store_tile_c<BM, BN, MS, OBF, EPI>(acc, g, m0, n0, smem);
    if (!more) break;
    __syncthreads();  // every wave is done with LDS (last MFMAs, epilogue reads)
    n_edge = n1 + BN > g.N;
    st.store(sA0, sB0, n_edge || (k_tail && kt_total == 1), o.b_cs);
    __syncthreads();
    t = t_next;
    m0 = m1;
    n0 = n1;
  }
}

template <int BM, int BN, int MS, bool OBF>
__global__ __launch_bounds__(64 * tile_waves(BM, BN)) void k_tile_pp(GemmArgs g) {
  persist_kernel<BM, BN, MS, OBF, false>(g);
}
template <int BM, int BN, int MS, bool OBF>
__global__ __launch_bounds__(64 * tile_waves(BM, BN)) void k_tile_pp_addmm(GemmArgs g) {
  persist_kernel<BM, BN, MS, OBF, true>(g);
}

// --------------------------------------------------------- grouped kernel
// One launch for all groups of a grouped product (an MoE layer's experts).
// The grid covers an upper bound of the row tiles (slots) times the column
// tiles; every workgroup derives its group and row tile from the device
// counts itself, so the host needs neither the counts nor a second kernel.

__device__ __forceinline__ int64_t uniform64(int64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Row ranges and row-tile counts of 64 consecutive groups, one per lane, as
// wave-wide inclusive prefix sums (rows_incl clamped by the caller).
template <int BM>
struct GroupChunk {
  int64_t lo, r;  // first row and row count of the lane's group
  int t, ts;      // row tiles of the lane's group, inclusive sum over the chunk
  int64_t rsum;   // rows of the whole chunk (unclamped)
  __device__ __forceinline__ void load(const GroupArgs& a, int c, int64_t row_base) {
    const int lane = threadIdx.x & 63;
    const int gi = c + lane;
    const int64_t cnt = gi < a.groups ? (int64_t)max(a.counts[gi], 0) : 0;
    int64_t p = cnt;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int64_t o = __shfl_up(p, d);
      if (lane >= d) p += o;
    }
    const int64_t hi = min(row_base + p, a.rows);
    lo = min(row_base + p - cnt, a.rows);
    r = hi - lo;
    t = (int)((r + BM - 1) / BM);
    ts = t;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int o = __shfl_up(ts, d);
      if (lane >= d) ts += o;
    }
    rsum = __shfl(p, 63);
  }
};

// Total row tiles of all groups.
template <int BM>
__device__ __forceinline__ int group_tiles_total(const GroupArgs& a, const GroupChunk<BM>& first) {
  int total = __shfl(first.ts, 63);
  int64_t row_base = min(first.rsum, a.rows);
  for (int c = 64; c < a.groups; c += 64) {
    GroupChunk<BM> k;
    k.load(a, c, row_base);
    total += __shfl(k.ts, 63);
    row_base = min(row_base + k.rsum, a.rows);
  }
  return total;
}

// Group, first row, row count and row tile of `slot`; false if the slot is
// past the last tile.
template <int BM>
__device__ __forceinline__ bool group_of_slot(const GroupArgs& a, const GroupChunk<BM>& first, int slot, int& grp,
                                              int64_t& row0, int64_t& rows_g, int& tm) {
  int tile_base = 0;
  int64_t row_base = 0;
  GroupChunk<BM> k = first;
  for (int c = 0; c < a.groups; c += 64) {
    if (c > 0) k.load(a, c, row_base);
    const uint64_t hit = __ballot(tile_base + k.ts > slot);
    if (hit) {
      const int f = __builtin_ctzll(hit);
      grp = c + f;
      row0 = __shfl(k.lo, f);
      rows_g = __shfl(k.r, f);
      tm = slot - (tile_base + __shfl(k.ts, f) - __shfl(k.t, f));
      return true;
    }
    tile_base += __shfl(k.ts, 63);
    row_base = min(row_base + k.rsum, a.rows);
  }
  return false;
}

template <int BM, int BN, int MS, int OUT, int DEPTH, bool EPI>
__device__ __forceinline__ void grouped_kernel(const GroupArgs& a) {
  typedef TileShape<BM, BN, MS> S;
  typedef typename AccOf<MS>::T Acc;
  __shared__ __attribute__((aligned(16))) char smem[S::SMEM];

  const int tiles_n = a.g.tiles_n;
  int t = blockIdx.x;
  int grp = 0, tm = 0, tn = 0;
  int64_t row0 = 0, rows_g = 0;
  if (a.counts == nullptr) {
    // strided batch: the grid is exactly groups x row tiles x column tiles
    if (a.g.swizzle) t = xcd_remap(t, (int)gridDim.x);
    const int slot = t / tiles_n;
    tn = t - slot * tiles_n;
    grp = slot / a.tiles_per_group;
    tm = slot - grp * a.tiles_per_group;
    rows_g = a.rows;
  } else {
    GroupChunk<BM> first;
    first.load(a, 0, 0);
    if (a.g.swizzle) {
      // XCD-aware order over the tiles that exist: each XCD takes a
      // contiguous range of (row tile, column tile) ids, the surplus blocks
      // leave
      const int n = group_tiles_total<BM>(a, first) * tiles_n;
      if (t >= n) return;
      t = xcd_remap(t, n);
    }
    const int slot = t / tiles_n;
    tn = t - slot * tiles_n;
    if (!group_of_slot<BM>(a, first, slot, grp, row0, rows_g, tm)) return;
  }
  // the same values in every lane: keep them scalar for the address bases
  grp = __builtin_amdgcn_readfirstlane(grp);
  tm = __builtin_amdgcn_readfirstlane(tm);
  row0 = uniform64(row0);
  rows_g = uniform64(rows_g);

  GemmArgs g = a.g;
  g.A += row0 * g.lda + (int64_t)grp * a.stride_a;
  g.B += (int64_t)grp * a.stride_b;
  g.C = static_cast<char*>(g.C) + (row0 * g.ldc + (int64_t)grp * a.stride_c) * (OUT == OUT_BF16 ? 2 : 4);
  if (EPI && g.bias != nullptr) g.bias += (int64_t)grp * a.stride_bias;
  g.M = rows_g;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const int kt_total = (int)((g.K + S::BK - 1) / S::BK);

  Acc acc[S::TM][S::TN];
#pragma unroll
  for (int i = 0; i < S::TM; ++i)
#pragma unroll
    for (int j = 0; j < S::TN; ++j) acc[i][j] = Acc{};

  tile_mainloop<BM, BN, MS, DEPTH>(g, m0, n0, 0, kt_total, acc, smem);
  store_tile_c<BM, BN, MS, OUT == OUT_BF16, EPI>(acc, g, m0, n0, smem);
}

// The grouped kernel, and its form with the AddMM epilogue (C_old and the
// bias row relative to each group's C).
template <int BM, int BN, int MS, int OUT, int DEPTH>
__global__ __launch_bounds__(64 * tile_waves(BM, BN)) void k_grouped(GroupArgs a) {
  grouped_kernel<BM, BN, MS, OUT, DEPTH, false>(a);
}
template <int BM, int BN, int MS, int OUT, int DEPTH>
__global__ __launch_bounds__(64 * tile_waves(BM, BN)) void k_grouped_addmm(GroupArgs a) {
  grouped_kernel<BM, BN, MS, OUT, DEPTH, true>(a);
}

// --------------------------------------------------------- stream-K kernel
// A persistent grid of g.grid workgroups. The first `sk_tiles` tiles (in
// tile-id order) are split into MAC iterations (one k-block each) and every
// workgroup takes `iters_per_wg` consecutive iterations. A tile covered by
// one workgroup is written to C directly; otherwise each piece goes to the
// tile's slot (workgroup - first workgroup of the tile) as a row-major fp32
// tile, summed later by k_sk_fixup. The remaining tiles are processed whole,
// data-parallel, by the grid.
template <int BM, int BN, int MS, bool OBF, bool EPI>
__device__ __forceinline__ void streamk_kernel(const GemmArgs& g) {
  typedef TileShape<BM, BN, MS> S;
  typedef typename AccOf<MS>::T Acc;
  __shared__ __attribute__((aligned(16))) char smem[S::SMEM];

  const int ntiles = g.tiles_m * g.tiles_n;
  const int ipt = (int)((g.K + S::BK - 1) / S::BK);
  const size_t tile_floats = (size_t)BM * BN;
  const int64_t total_sk = (int64_t)g.sk_tiles * ipt;

  int64_t it = (int64_t)blockIdx.x * g.iters_per_wg;
  const int64_t it_end = min(it + (int64_t)g.iters_per_wg, total_sk);
  while (it < it_end) {
    const int tile = (int)(it / ipt);
    const int k_begin = (int)(it - (int64_t)tile * ipt);
    const int k_end = (int)min((int64_t)ipt, k_begin + (it_end - it));
    int tm, tn;
    tile_coords(tile, g.tiles_m, g.tiles_n, g.swizzle, tm, tn);
    const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
    Acc acc[S::TM][S::TN];
#pragma unroll
    for (int i = 0; i < S::TM; ++i)
#pragma unroll
      for (int j = 0; j < S::TN; ++j) acc[i][j] = Acc{};
    __syncthreads();
    tile_mainloop<BM, BN, MS, streamk_depth(BM, BN)>(g, m0, n0, k_begin, k_end, acc, smem);
    const int64_t t0 = (int64_t)tile * ipt;
    const int first_wg = (int)(t0 / g.iters_per_wg);
    const int last_wg = (int)min((int64_t)g.grid - 1, (t0 + ipt - 1) / g.iters_per_wg);
    if (first_wg == last_wg) {
      store_tile_c<BM, BN, MS, OBF, EPI>(acc, g, m0, n0, smem);
    } else {
      float* slot = g.ws + ((size_t)tile * g.ws_pk + (blockIdx.x - first_wg)) * tile_floats;
      store_acc_f32<BM, BN, MS>(acc, slot, BN, 0, 0, BM, BN);
    }
    it += k_end - k_begin;
  }

  for (int tile = g.sk_tiles + blockIdx.x; tile < ntiles; tile += g.grid) {
    int tm, tn;
    tile_coords(tile, g.tiles_m, g.tiles_n, g.swizzle, tm, tn);
    const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
    Acc acc[S::TM][S::TN];
#pragma unroll
    for (int i = 0; i < S::TM; ++i)
#pragma unroll
      for (int j = 0; j < S::TN; ++j) acc[i][j] = Acc{};
    __syncthreads();
    tile_mainloop<BM, BN, MS, streamk_depth(BM, BN)>(g, m0, n0, 0, ipt, acc, smem);
    store_tile_c<BM, BN, MS, OBF, EPI>(acc, g, m0, n0, smem);
  }
}

template <int BM, int BN, int MS, bool OBF>
__global__ __launch_bounds__(64 * tile_waves(BM, BN)) void k_streamk(GemmArgs g) {
  streamk_kernel<BM, BN, MS, OBF, false>(g);
}
template <int BM, int BN, int MS, bool OBF>
__global__ __launch_bounds__(64 * tile_waves(BM, BN)) void k_streamk_addmm(GemmArgs g) {
  streamk_kernel<BM, BN, MS, OBF, true>(g);
}

// Sums the pieces of every split stream-K tile in workgroup order and writes
// C. Grid: (sk_tiles, chunks); a thread handles 8 consecutive columns of a
// tile row.
template <bool OBF>
__global__ __launch_bounds__(256) void k_sk_fixup(GemmArgs g, int BM, int BN) {
  const int tile = blockIdx.x;
  const int ipt = (int)((g.K + 63) / 64);
  const int64_t t0 = (int64_t)tile * ipt;
  const int first_wg = (int)(t0 / g.iters_per_wg);
  const int last_wg = (int)min((int64_t)g.grid - 1, (t0 + ipt - 1) / g.iters_per_wg);
  if (first_wg == last_wg) return;  // written directly by its workgroup
  const int pieces = last_wg - first_wg + 1;
  int tm, tn;
  tile_coords(tile, g.tiles_m, g.tiles_n, g.swizzle, tm, tn);
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const size_t tile_floats = (size_t)BM * BN;
  const float* base = g.ws + (size_t)tile * g.ws_pk * tile_floats;
  const int gpr = BN / 8;
  for (int e = blockIdx.y * 256 + threadIdx.x; e < BM * gpr; e += gridDim.y * 256) {
    const int row = e / gpr, c0 = (e % gpr) * 8;
    const int64_t gr = m0 + row, gc = n0 + c0;
    if (gr >= g.M || gc >= g.N) continue;
    const float* src = base + (size_t)row * BN + c0;
    f32x4 s0 = *reinterpret_cast<const f32x4*>(src), s1 = *reinterpret_cast<const f32x4*>(src + 4);
    for (int p = 1; p < pieces; ++p) {
      s0 += *reinterpret_cast<const f32x4*>(src + p * tile_floats);
      s1 += *reinterpret_cast<const f32x4*>(src + p * tile_floats + 4);
    }
    const float v[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
    store_out8<OBF>(g, gr, gc, v, g.N - gc);
  }
}

// -------------------------------------------------- split-K reduction kernel
// C = sum over p = 0 .. P_k - 1 of the row-major fp32 slices ws[p] (M x ldw,
// ldw a multiple of 8). A thread handles 8 columns of a row; when there are
// few outputs and many partitions, G = 2^lg threads share one group of 8
// columns: thread j sums the contiguous partitions [j*P_k/G, (j+1)*P_k/G) in
// ascending order and the G sums are added in a fixed pairwise tree through
// LDS. The order depends only on (P_k, G), never on timing.
template <bool OBF>
__global__ __launch_bounds__(256) void k_reduce(GemmArgs g, int lg) {
  __shared__ f32x4 red[2][256];
  const int G = 1 << lg, EB = 256 >> lg;
  const int t = threadIdx.x, el = t & (EB - 1), j = t >> (8 - lg);
  const int64_t gpr = (g.N + 7) / 8;
  const int64_t e = (int64_t)blockIdx.x * EB + el;
  const bool live = e < g.M * gpr;
  const int64_t row = live ? e / gpr : 0, c0 = live ? (e - row * gpr) * 8 : 0;
  const size_t slice = (size_t)g.M * (size_t)g.ldw;
  const float* src = g.ws + row * g.ldw + c0;
  const int p0 = (int)(((int64_t)j * g.pk) >> lg), p1 = (int)(((int64_t)(j + 1) * g.pk) >> lg);
  f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = s0;
  if (live && p0 < p1) {
    s0 = *reinterpret_cast<const f32x4*>(src + p0 * slice);
    s1 = *reinterpret_cast<const f32x4*>(src + p0 * slice + 4);
    for (int p = p0 + 1; p < p1; ++p) {
      s0 += *reinterpret_cast<const f32x4*>(src + p * slice);
      s1 += *reinterpret_cast<const f32x4*>(src + p * slice + 4);
    }
  }
  if (lg > 0) {
    // pairwise tree over j: at step h, thread j (a multiple of 2h) adds j + h
    red[0][t] = s0;
    red[1][t] = s1;
    __syncthreads();
    for (int h = 1; h < G; h <<= 1) {
      if ((j & (2 * h - 1)) == 0) {
        s0 += red[0][t + h * EB];
        s1 += red[1][t + h * EB];
        red[0][t] = s0;
        red[1][t] = s1;
      }
      __syncthreads();
    }
  }
  if (!live || j != 0) return;
  const float v[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
  store_out8<OBF>(g, row, c0, v, g.N - c0);
}

// -------------------------------------------------------- skinny-M kernel
// C (M x N, M <= 16*MT) = A * B with B streamed once. A wave owns 128
// columns: lane l loads, for k-group l/16, an 8 x 8 block (8 k-rows, 8
// columns starting at 8*(l%16)), transposes it in registers and issues one
// 16x16x32 MFMA per column j, so MFMA j computes the 16 columns
// {base + 8c + j}. A fragments (16 rows x 32 k) come straight from global
// memory (A is small and stays in cache). WKW waves of a workgroup split the
// workgroup's k-range and are reduced through LDS in wave order.
// BT: B stored column-major (element (k, j) at B[j * ldb + k]). A column's 8
// consecutive k are then contiguous, which is the MFMA's B fragment: each of
// the 8 columns is one 16-byte load (like an A fragment) and no register
// transpose is needed.
template <int MT, int WKW, bool OBF, bool BT>
__device__ __forceinline__ void skinny_m_kernel(const GemmArgs& g) {
  constexpr int WNW = 4 / WKW;
  constexpr int NB = 128 * WNW;
  constexpr int U = 2;
  constexpr int NV = MT * 8;  // f32x4 accumulators per lane
  __shared__ f32x4 red[WKW > 1 ? (WKW - 1) * WNW * NV * 64 : 1];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wc = wave % WNW, wk = wave / WNW;
  const int cb = blockIdx.x, split = blockIdx.y;
  const int64_t M = g.M, N = g.N, K = g.K, lda = g.lda, ldb = g.ldb;
  const int64_t col0 = (int64_t)cb * NB + wc * 128 + 8 * (lane & 15);
  const int kg = lane >> 4;
  const int kb_total = (int)((K + 31) / 32);
  const int kb0 = min(split * g.kper, kb_total);
  const int kb1 = min(kb0 + g.kper, kb_total);
  const bool k_tail = (K % 32) != 0;
  const bool n_edge = (int64_t)(cb + 1) * NB > N;

  f32x4 acc[MT][8];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t nvalid = N - col0;
  // Straight-line loads: the lane's 8 columns start at min(col0, N - 8) (never
  // past the row end) and the leading extra columns are dropped afterwards;
  // B rows past K are clamped and dropped; A vectors of the K tail end at the
  // row end. K < 8 or N < 8 take element loads instead.
  const bool small = BT ? K < 8 : (K < 8 || N < 8);
  const int64_t cst = (small || BT) ? col0 : min(col0, N - 8);
  const int cs = small ? 0 : (int)min(col0 - cst, (int64_t)8);
  for (int kb = kb0 + wk; kb < kb1; kb += WKW * U) {
    u32x4 rb[U][8];
    u32x4 fa[U][MT];
    uint32_t past[U];
    int sa[U];
    bool edge = n_edge;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kbu = kb + u * WKW;
      const int64_t k = (int64_t)kbu * 32 + kg * 8;
      const bool on = kbu < kb1;  // uniform over the wave
      edge = edge || !on || (k_tail && kbu == kb_total - 1);
      past[u] = 0;
      if (BT) {
        // column j of the lane: col0 + j, clamped into the matrix (columns
        // past N compute values that are never stored)
        const int64_t st = small ? k : min(k, K - 8);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const uint16_t* bc = g.B + min(col0 + j, N - 1) * ldb;
          if (!small) {
            rb[u][j] = load16(bc + st);
          } else {
            const u32x4 v = load_row8_small(bc, k, K);
            rb[u][j] = on ? v : u32x4{0u, 0u, 0u, 0u};
          }
        }
      }
      if (!small) {
        if (!BT) {
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            rb[u][i] = load16(g.B + min(k + i, K - 1) * ldb + cst);
            past[u] |= (uint32_t)(!on || k + i >= K) << i;
          }
        }
        const int64_t st = min(k, K - 8);
        sa[u] = on ? (int)min(k - st, (int64_t)8) : 8;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int64_t row = min((int64_t)(mt * 16 + (lane & 15)), M - 1);
          fa[u][mt] = load16(g.A + row * lda + st);
        }
      } else {
        sa[u] = 0;
        if (!BT) {
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const u32x4 v = load_row8_small(g.B + min(k + i, K - 1) * ldb, col0, N);
            rb[u][i] = (on && k + i < K) ? v : u32x4{0u, 0u, 0u, 0u};
          }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const int64_t row = min((int64_t)(mt * 16 + (lane & 15)), M - 1);
          const u32x4 v = load_row8_small(g.A + row * lda, k, K);
          fa[u][mt] = on ? v : u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (edge && !small) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
          rb[u][i] = shift_down(rb[u][i], BT ? sa[u] : (((past[u] >> i) & 1) ? 8 : cs));
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) fa[u][mt] = shift_down(fa[u][mt], sa[u]);
      }
      u32x4 col[8];
      if constexpr (BT) {
#pragma unroll
        for (int j = 0; j < 8; ++j) col[j] = rb[u][j];
      } else {
        transpose8x8(rb[u], col);
      }
#pragma unroll
      for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[mt][j] = mfma16(fa[u][mt], col[j], acc[mt][j]);
    }
  }

  if constexpr (WKW > 1) {
    if (wk > 0) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 8; ++j) red[(((wk - 1) * WNW + wc) * NV + mt * 8 + j) * 64 + lane] = acc[mt][j];
    }
    __syncthreads();
    if (wk != 0) return;
    for (int w = 1; w < WKW; ++w)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[mt][j] += red[(((w - 1) * WNW + wc) * NV + mt * 8 + j) * 64 + lane];
  }
  if (nvalid <= 0) return;

  // Output: lane holds rows mt*16 + 4*(l/16) + r, columns col0 .. col0+7.
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = mt * 16 + (lane >> 4) * 4 + r;
      if (row < M) {
        float o[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] = acc[mt][j][r];
        if (g.pk == 1)
          store_out8<OBF>(g, row, col0, o, nvalid);
        else
          store_c8<false>(g.ws + (size_t)split * (size_t)M * (size_t)g.ldw, row * g.ldw + col0, o, nvalid);
      }
    }
}

template <int MT, int WKW, bool OBF>
__global__ __launch_bounds__(256) void k_skinny_m(GemmArgs g) {
  skinny_m_kernel<MT, WKW, OBF, false>(g);
}
template <int MT, int WKW, bool OBF>
__global__ __launch_bounds__(256) void k_skinny_m_bt(GemmArgs g) {
  skinny_m_kernel<MT, WKW, OBF, true>(g);
}

// -------------------------------------------------------- skinny-N kernel
// C (M x N, N <= 16*NT) = A * B with A streamed once. The workgroup walks its
// k-range in chunks of at most SKN_KMAX: each chunk of B is transposed into
// LDS (B is small and comes from cache), then each wave streams 16*RB rows
// of A over the chunk, one 16-byte fragment per lane per 32-k block, and
// issues RB*NT 16x16x32 MFMAs against the resident B fragments.
constexpr int SKN_KMAX = 512;

template <int NT, int RB, bool OBF>
__global__ __launch_bounds__(256) void k_skinny_n(GemmArgs g) {
  constexpr int NCOL = NT * 16;
  constexpr int KCH = SKN_KMAX / 8;  // 16-byte chunks per LDS row
  constexpr int CKB = SKN_KMAX / 32; // 32-k blocks per chunk
  constexpr int U = 2;
  __shared__ u32x4 sBt[NCOL * KCH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rbk = blockIdx.x, split = blockIdx.y;
  const int64_t M = g.M, N = g.N, K = g.K, lda = g.lda, ldb = g.ldb;
  const int kb_total = (int)((K + 31) / 32);
  const int kb0 = min(split * g.kper, kb_total);
  const int kb1 = min(kb0 + g.kper, kb_total);
  const bool k_tail = (K % 32) != 0;

  f32x4 acc[RB][NT];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[rb][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t row0 = (int64_t)rbk * (64 * RB) + wave * (16 * RB) + (lane & 15);
  const int kg = lane >> 4;
  const bool small = K < 8;
  for (int cb0 = kb0; cb0 < kb1; cb0 += CKB) {
    const int cb1 = min(cb0 + CKB, kb1);
    const int64_t kbeg = (int64_t)cb0 * 32;
    const int nkc = (cb1 - cb0) * 4;  // 8-k chunks of this chunk
    if (cb0 != kb0) __syncthreads();  // every wave is done with the previous chunk
    // Stage B^T: block (kc, ng) = rows kbeg + 8kc .. +7, columns 8ng .. 8ng+7.
    for (int blk = tid; blk < nkc * (NCOL / 8); blk += 256) {
      const int ng = blk % (NCOL / 8), kc = blk / (NCOL / 8);
      const int64_t n = (int64_t)ng * 8;
      u32x4 r[8], c[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int64_t k = kbeg + kc * 8 + i;
        const u32x4 v = load_row(g.B + min(k, K - 1) * ldb, n, N);
        r[i] = k < K ? v : u32x4{0u, 0u, 0u, 0u};
      }
      transpose8x8(r, c);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int nn = ng * 8 + j;
        sBt[nn * KCH + (kc ^ (nn & 15))] = c[j];
      }
    }
    __syncthreads();

    for (int kb = cb0; kb < cb1; kb += U) {
      u32x4 fa[U][RB];
      int sa[U];
      bool edge = false;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t k = (int64_t)(kb + u) * 32 + kg * 8;
        const bool on = kb + u < cb1;  // uniform
        edge = edge || !on || (k_tail && kb + u == kb_total - 1);
        if (!small) {
          // the K tail's vectors end at the row end; leading extras dropped below
          const int64_t st = min(k, K - 8);
          sa[u] = on ? (int)min(k - st, (int64_t)8) : 8;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) fa[u][rb] = load16(g.A + min(row0 + rb * 16, M - 1) * lda + st);
        } else {
          sa[u] = 0;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            const u32x4 v = load_row8_small(g.A + min(row0 + rb * 16, M - 1) * lda, k, K);
            fa[u][rb] = on ? v : u32x4{0u, 0u, 0u, 0u};
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (kb + u >= cb1) break;
        if (edge && !small) {
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) fa[u][rb] = shift_down(fa[u][rb], sa[u]);
        }
        const int kc = (kb + u - cb0) * 4 + kg;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int nn = nt * 16 + (lane & 15);
          const u32x4 fb = sBt[nn * KCH + (kc ^ (nn & 15))];
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) acc[rb][nt] = mfma16(fa[u][rb], fb, acc[rb][nt]);
        }
      }
    }
  }

  // Output: lane holds column nt*16 + l%16 of rows base + rb*16 + 4*(l/16) + r.
  const int64_t rbase = (int64_t)rbk * (64 * RB) + wave * (16 * RB) + (lane >> 4) * 4;
  float* part = g.ws + (size_t)split * (size_t)M * (size_t)g.ldw;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int64_t col = nt * 16 + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = rbase + rb * 16 + r;
        if (row < M && col < N) {
          if (g.pk == 1)
            store_out<OBF>(g, row, col, acc[rb][nt][r]);
          else
            part[row * g.ldw + col] = acc[rb][nt][r];
        }
      }
    }
}

// -------------------------------------------------------- small-K kernel
// K <= KMAX (8 or 16): C is a rank-K update, bound by writing C once. A
// thread owns 8 columns and a run of R = g.kper rows (a multiple of 4): it
// keeps the K x 8 block of B it needs in registers, then for each group of 4
// rows loads the 4 A rows (K values each), forms the 4 x 8 outputs with fp32
// FMAs in ascending k and stores them as 16-byte (bf16) or 32-byte (fp32)
// row segments. Thread t takes column group t % ceil(N/8) and row run
// t / ceil(N/8), so neighbouring threads write neighbouring segments of a
// row; B is read once per R rows, the A rows are shared by the threads of a
// row run.
template <int KMAX, bool OBF>
__global__ __launch_bounds__(256) void k_smallk(GemmArgs g) {
  const int64_t M = g.M, N = g.N, K = g.K;
  const int64_t R = g.kper;
  const int64_t ncg = (N + 7) / 8;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= ncg * ((M + R - 1) / R)) return;
  const int64_t rg = t / ncg, cg = t - rg * ncg;
  const int64_t r0 = rg * R, c0 = cg * 8;
  const int64_t rend = min(r0 + R, M);

  // B rows 0..K-1, columns c0..c0+7 (zeros past N, rows past K zero)
  float b[KMAX][8];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (k < K) v = load_row(g.B + (int64_t)k * g.ldb, c0, N);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      b[k][2 * e] = from16(v[e] & 0xFFFFu);
      b[k][2 * e + 1] = from16(v[e] >> 16);
    }
  }
  for (int64_t rb = r0; rb < rend; rb += 4) {
    // the 4 A rows of this group as raw 16-bit values (rows past M repeat row M-1)
    u32x4 av[4][KMAX / 8];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = min(rb + r, M - 1);
#pragma unroll
      for (int h = 0; h < KMAX / 8; ++h) av[r][h] = load_row(g.A + row * g.lda, h * 8, K);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float acc[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = 0.f;
#pragma unroll
      for (int k = 0; k < KMAX; ++k) {
        const uint32_t w = av[r][k / 8][(k % 8) / 2];
        const float a = from16((k & 1) ? (w >> 16) : (w & 0xFFFFu));
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = __builtin_fmaf(a, b[k][j], acc[j]);
      }
      if (rb + r < rend) store_out8<OBF>(g, rb + r, c0, acc, N - c0);
    }
  }
}

// Wide rows (the plan's tile_n = SMALLK_WIN_COLS): a workgroup owns a band of
// R = g.kper rows and SMALLK_WIN_COLS columns, and per row writes the window
// of the same width that starts at the 128-byte line boundary at or before
// its first column. The windows of a row then tile it line by line, and no
// line of C is written by two workgroups (but a row's first and last). A
// line that two workgroups write in parts -- on different CUs, usually on
// different XCDs -- is written back to memory twice in parts, and such
// writes cost several times a whole line: with misaligned row starts, a
// 16-byte-per-lane store pattern wrote at about 3.4 TB/s against 5.3 TB/s
// for the same bytes in line-aligned rows. The window reaches up to 63
// columns to the left of the workgroup's own, so every thread computes 8
// columns of a range that starts 64 columns before them (256 threads: 64
// halo + SMALLK_WIN_COLS columns). Groups of rows go through LDS in C's
// format (after the AddMM epilogue) and are stored from there, shifted to
// the window, as whole 16-byte (bf16) or 32-byte (fp32) segments. The sums
// run over pairs of k in ascending order with the packed two-term dot
// product (fp32 accumulator; half the instructions of single FMAs, which
// bound this kernel on K > 4); pairs past K are skipped. The epilogue reads
// C_old at every computed column; the halo columns outside the window
// belong to the neighbouring workgroup, and their values are never stored.
template <int KMAX, bool OBF>
__global__ __launch_bounds__(256) void k_smallk_win(GemmArgs g) {
  constexpr int H = KMAX / 8, RG = OBF ? 4 : 2;  // 16-byte chunks of an A row; rows per LDS round
  constexpr int LE = OBF ? 64 : 32;     // elements of C per 128-byte line
  constexpr int SW = OBF ? 4 : 8;       // dwords of a thread's 8 outputs
  __shared__ u32x4 sA[SMALLK_MAX_ROWS * H];
  __shared__ uint32_t sC[2][RG][256 * SW + 4];
  const int tid = threadIdx.x;
  const int64_t M = g.M, N = g.N, K = g.K, R = g.kper;
  const int64_t c_own = (int64_t)blockIdx.x * SMALLK_WIN_COLS;
  const int64_t c0 = c_own - 64 + 8 * tid;  // this thread's 8 computed columns
  const int valid = c0 < 0 ? 0 : (int)min((int64_t)8, N - c0);
  const int64_t r0 = (int64_t)blockIdx.y * R, r1 = min(r0 + R, M);
  for (int64_t i = tid; i < (r1 - r0) * H; i += 256)
    sA[i] = load_row(g.A + (r0 + i / H) * g.lda, (i % H) * 8, K);
  // B rows 2i and 2i+1 of column j packed into one word (rows past K zero)
  uint32_t bp[KMAX / 2][8];
#pragma unroll
  for (int i = 0; i < KMAX / 2; ++i) {
    u32x4 v0 = u32x4{0u, 0u, 0u, 0u}, v1 = v0;
    if (2 * i < K && valid > 0) v0 = load_row(g.B + (int64_t)(2 * i) * g.ldb, c0, N);
    if (2 * i + 1 < K && valid > 0) v1 = load_row(g.B + (int64_t)(2 * i + 1) * g.ldb, c0, N);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      bp[i][2 * e] = __builtin_amdgcn_perm(v1[e], v0[e], 0x05040100u);      // low halves
      bp[i][2 * e + 1] = __builtin_amdgcn_perm(v1[e], v0[e], 0x07060302u);  // high halves
    }
  }
  __syncthreads();
  for (int64_t rb = r0; rb < r1; rb += RG) {
    const int par = (int)(((rb - r0) / RG) & 1);
#pragma unroll
    for (int r = 0; r < RG; ++r) {
      const int64_t row = min(rb + r, r1 - 1);
      const u32x4* a_row = sA + (row - r0) * H;
      float acc[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = 0.f;
#pragma unroll
      for (int i = 0; i < KMAX / 2; ++i) {
        if (2 * i < K) {  // (uniform)
          const uint32_t w = a_row[i / 4][i % 4];  // A elements 2i, 2i+1 of the row
#pragma unroll
          for (int j = 0; j < 8; ++j) acc[j] = dot2(w, bp[i][j], acc[j]);
        }
      }
      epi_apply<OBF, 8>(g, acc, row, c0, valid);
      uint32_t* dst = &sC[par][r][SW * tid];
      if constexpr (OBF) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = (uint32_t)to16(acc[2 * e]) | ((uint32_t)to16(acc[2 * e + 1]) << 16);
        *reinterpret_cast<u32x4*>(dst) = w;
      } else {
        *reinterpret_cast<f32x4*>(dst) = f32x4{acc[0], acc[1], acc[2], acc[3]};
        *reinterpret_cast<f32x4*>(dst + 4) = f32x4{acc[4], acc[5], acc[6], acc[7]};
      }
    }
    __syncthreads();
    if (tid < SMALLK_WIN_COLS / 8) {
#pragma unroll
      for (int r = 0; r < RG; ++r) {
        const int64_t row = rb + r;
        if (row >= r1) break;
        const int64_t rowoff = row * g.ldc;
        // elements of C between the line boundary and the first own column
        const int mu = (int)(((uintptr_t)g.C / (OBF ? 2 : 4) + rowoff + c_own) & (LE - 1));
        const int o = 64 - mu + 8 * tid;  // offset of the window chunk in the computed range: 1 .. 2040
        const int64_t col = c_own - mu + 8 * tid;
        const uint32_t* src = &sC[par][r][0];
        uint32_t y[SW];
        if constexpr (OBF) {
          const int d0 = o >> 1;
          if (o & 1) {  // odd element offset: funnel pairs of dwords by 2 bytes
            uint32_t x[5];
#pragma unroll
            for (int d = 0; d < 5; ++d) x[d] = src[d0 + d];
#pragma unroll
            for (int d = 0; d < 4; ++d) y[d] = __builtin_amdgcn_alignbyte(x[d + 1], x[d], 2);
          } else {
#pragma unroll
            for (int d = 0; d < 4; ++d) y[d] = src[d0 + d];
          }
        } else {
#pragma unroll
          for (int d = 0; d < 8; ++d) y[d] = src[o + d];
        }
        if (col >= 0 && col + 8 <= N) {
          if constexpr (OBF) {
            const u32x4 w = u32x4{y[0], y[1], y[2], y[3]};
            __builtin_memcpy(static_cast<uint16_t*>(g.C) + rowoff + col, &w, 16);
          } else {
            float* p = static_cast<float*>(g.C) + rowoff + col;
            const u32x4 w0 = u32x4{y[0], y[1], y[2], y[3]}, w1 = u32x4{y[4], y[5], y[6], y[7]};
            __builtin_memcpy(p, &w0, 16);
            __builtin_memcpy(p + 4, &w1, 16);
          }
        } else {
          for (int e = 0; e < 8; ++e) {
            if (col + e < 0 || col + e >= N) continue;
            if constexpr (OBF)
              static_cast<uint16_t*>(g.C)[rowoff + col + e] = (uint16_t)(y[e >> 1] >> (16 * (e & 1)));
            else
              static_cast<uint32_t*>(g.C)[rowoff + col + e] = y[e];
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------- direct kernel
// Latency-lean kernel for small problems: no LDS staging, no register
// transposes. A wave computes one 32 x 32 block of C with 32x32x16 MFMAs,
// reading its operand fragments straight from global memory (they come from
// cache): lane l takes row l % 32 of A and column l % 32 of B, k-group l / 32
// (8 consecutive k). The A fragment is one 16-byte load; the B fragment is 8
// two-byte loads down the column. B is passed as the MFMA's first operand, so
// the accumulators hold the transposed block: one row of C per lane, in runs
// of four consecutive columns (8- or 16-byte stores). Rows past M and columns past N are clamped
// (their results are never stored); k past K reads as zero. WK = 1: the four
// waves cover a 64 x 64 block of C, each over all of K. WK = 4 or 16: the WK
// waves split the 32-k blocks of one 32 x 32 block evenly and wave 0 adds
// the partial sums in wave order through LDS (a partition of one block is
// wave 0's alone, and the others leave at once).
template <int WK, int OUT>
__global__ __launch_bounds__(WK == 1 ? 256 : 64 * WK) void k_direct(GemmArgs g) {
  constexpr int U = 4;  // 32-k blocks whose loads are issued together
  __shared__ f32x16 red[WK > 1 ? (WK - 1) * 64 : 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t M = g.M, N = g.N, K = g.K;
  const int tm = blockIdx.x / g.tiles_n, tn = blockIdx.x - tm * g.tiles_n;
  int64_t m0, n0;
  int kb0, kb1;
  const int kb_total = (int)((K + 31) / 32);
  // this workgroup's K partition (P_k > 1: blockIdx.y of g.pk, g.kper blocks)
  const int split = blockIdx.y;
  const int pb0 = min(split * g.kper, kb_total), pb1 = min(pb0 + g.kper, kb_total);
  if constexpr (WK == 1) {
    m0 = (int64_t)tm * 64 + (wave >> 1) * 32;
    n0 = (int64_t)tn * 64 + (wave & 1) * 32;
    kb0 = pb0;
    kb1 = pb1;
  } else {
    m0 = (int64_t)tm * 32;
    n0 = (int64_t)tn * 32;
    const int per = (pb1 - pb0 + WK - 1) / WK;
    kb0 = min(pb0 + wave * per, pb1);
    kb1 = min(kb0 + per, pb1);
  }
  const int kg = lane >> 5;
  const int64_t lda = g.lda, ldb = g.ldb;
  // Loads take a wave-uniform base (row m0 of A, row k of B) plus a per-lane
  // 32-bit byte offset (the host keeps lda, ldb < 2^23), so the address
  // arithmetic runs on the scalar unit.
  // (A's base row is clamped like the lanes' rows: a wave of the 64 x 64
  // layout can start past M, and the offsets must stay non-negative.)
  const int64_t ma = min(m0, M - 1);
  const uint32_t a_off = (uint32_t)(((min(m0 + (lane & 31), M - 1) - ma) * lda + kg * 8) * 2);
  const uint32_t b_off = (uint32_t)((min(n0 + (lane & 31), N - 1) + (int64_t)kg * 8 * ldb) * 2);
  const uint16_t* A0 = g.A + ma * lda;

  f32x16 acc = {};
  // whole 32-k blocks: no k checks
  const int kbf = min(kb1, (int)(K / 32));
  int kb = kb0;
  auto block = [&](int kbk, u32x4 (&a)[2], u32x4 (&b)[2]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t k = (int64_t)kbk * 32 + h * 16;
      a[h] = load16(at(A0 + k, a_off));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t lo = *at(g.B + (k + 2 * e) * ldb, b_off);
        const uint32_t hi = *at(g.B + (k + 2 * e + 1) * ldb, b_off);
        b[h][e] = lo | (hi << 16);
      }
    }
  };
  for (; kb + U <= kbf; kb += U) {
    u32x4 a[U][2], b[U][2];
#pragma unroll
    for (int u = 0; u < U; ++u) block(kb + u, a[u], b[u]);
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int h = 0; h < 2; ++h) acc = mfma32(b[u][h], a[u][h], acc);
  }
  for (; kb < kbf; ++kb) {
    u32x4 a[2], b[2];
    block(kb, a, b);
#pragma unroll
    for (int h = 0; h < 2; ++h) acc = mfma32(b[h], a[h], acc);
  }
  const uint16_t* pa = g.A + min(m0 + (lane & 31), M - 1) * lda + kg * 8;
  const uint16_t* pb = g.B + min(n0 + (lane & 31), N - 1) + (int64_t)kg * 8 * ldb;
  // the partial last 32-k block (if this wave owns it): element loads, zero past K
  if (kb < kb1) {
    const int64_t kbase = (int64_t)kb * 32 + kg * 8;
    const uint16_t* ra = pa - kg * 8;
    const uint16_t* cb = pb - (int64_t)kg * 8 * ldb;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      u32x4 a, b;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        // clamped loads are always in bounds; issue them unconditionally and
        // zero the values past K afterwards
        const int64_t k0 = kbase + h * 16 + 2 * e, k1 = k0 + 1;
        const int64_t c0 = min(k0, K - 1), c1 = min(k1, K - 1);
        const uint32_t va0 = ra[c0], va1 = ra[c1], vb0 = cb[c0 * ldb], vb1 = cb[c1 * ldb];
        a[e] = (k0 < K ? va0 : 0u) | ((k1 < K ? va1 : 0u) << 16);
        b[e] = (k0 < K ? vb0 : 0u) | ((k1 < K ? vb1 : 0u) << 16);
      }
      acc = mfma32(b, a, acc);
    }
  }

  if constexpr (WK > 1) {
    if (pb1 - pb0 <= 1) {
      // (uniform over the workgroup) at most one 32-k block: wave 0 holds
      // the whole sum and the other waves have none to add
      if (wave != 0) return;
    } else {
      if (wave > 0) red[(wave - 1) * 64 + lane] = acc;
      __syncthreads();
      if (wave != 0) return;
#pragma unroll
      for (int w = 1; w < WK; ++w) acc += red[(w - 1) * 64 + lane];
    }
  }
  // (operands swapped: the MFMA forms the transposed block) the lane holds
  // row m0 + lane % 32 and, for q = 0..3, the four consecutive columns
  // n0 + 8q + 4 * (lane / 32) .. +3
  // Wide outputs over many workgroups are bound by writing C: the 64 x 64
  // configuration then sends its block through LDS (rows padded by 4
  // elements) so that it leaves as whole 16-byte row segments. Small grids
  // are bound by latency and store straight from the registers.
  if (WK == 1 && N >= 64 && gridDim.x * gridDim.y >= 256) {
    typedef typename std::conditional<OUT == OUT_BF16, uint16_t, float>::type T;
    constexpr int LD = 64 + 4, VEC = 16 / sizeof(T);  // elements per 16-byte chunk
    __shared__ __attribute__((aligned(16))) T ct[64 * LD];
    const int r = (wave >> 1) * 32 + (lane & 31);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c = (wave & 1) * 32 + 8 * q + 4 * (lane >> 5);
      float w[4] = {acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]};
      if constexpr (OUT != OUT_PARTIAL) {
        const int64_t gr = (int64_t)tm * 64 + r, gc = (int64_t)tn * 64 + c;
        if (g.epi && gr < M && gc < N) epi_apply<OUT == OUT_BF16, 4>(g, w, gr, gc, N - gc);
      }
      if constexpr (OUT == OUT_BF16) {
        const uint32_t lo = (uint32_t)to16(w[0]) | ((uint32_t)to16(w[1]) << 16);
        const uint32_t hi = (uint32_t)to16(w[2]) | ((uint32_t)to16(w[3]) << 16);
        *reinterpret_cast<uint64_t*>(ct + r * LD + c) = (uint64_t)lo | ((uint64_t)hi << 32);
      } else {
        const f32x4 v = {w[0], w[1], w[2], w[3]};
        *reinterpret_cast<f32x4*>(ct + r * LD + c) = v;
      }
    }
    __syncthreads();
    const int64_t tm0 = (int64_t)tm * 64, tn0 = (int64_t)tn * 64;
    T* dst = OUT == OUT_PARTIAL ? reinterpret_cast<T*>(g.ws + (size_t)split * (size_t)M * (size_t)g.ldw)
                                : static_cast<T*>(g.C);
    const int64_t ldd = OUT == OUT_PARTIAL ? g.ldw : g.ldc;
    constexpr int CPR = 64 / VEC;  // chunks per row
    for (int e = threadIdx.x; e < 64 * CPR; e += 256) {
      const int rr = e / CPR, cc = (e % CPR) * VEC;
      const int64_t gr = tm0 + rr, gc = tn0 + cc;
      if (gr >= M || gc >= N) continue;
      const T* src = ct + rr * LD + cc;  // 8-byte aligned
      T* d = dst + gr * ldd + gc;
      if (gc + VEC <= N) {
        const uint64_t v[2] = {*reinterpret_cast<const uint64_t*>(src),
                               *reinterpret_cast<const uint64_t*>(src + VEC / 2)};
        __builtin_memcpy(d, v, 16);
      } else {
        for (int j = 0; j < (int)(N - gc); ++j) d[j] = src[j];
      }
    }
    return;
  }
  const int64_t row = m0 + (lane & 31);
  if (row >= M) return;
  float* part = g.ws + (size_t)split * (size_t)M * (size_t)g.ldw;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t col = n0 + 8 * q + 4 * (lane >> 5);
    float v[4] = {acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]};
    if constexpr (OUT != OUT_PARTIAL)
      if (g.epi && col < N) epi_apply<OUT == OUT_BF16, 4>(g, v, row, col, N - col);
    if (col + 4 <= N) {
      if constexpr (OUT == OUT_PARTIAL) {
        __builtin_memcpy(part + row * g.ldw + col, v, 16);
      } else if constexpr (OUT == OUT_BF16) {
        const uint32_t lo = (uint32_t)to16(v[0]) | ((uint32_t)to16(v[1]) << 16);
        const uint32_t hi = (uint32_t)to16(v[2]) | ((uint32_t)to16(v[3]) << 16);
        const uint64_t w = (uint64_t)lo | ((uint64_t)hi << 32);
        __builtin_memcpy(static_cast<uint16_t*>(g.C) + row * g.ldc + col, &w, 8);
      } else {
        __builtin_memcpy(static_cast<float*>(g.C) + row * g.ldc + col, v, 16);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (col + e >= N) break;
        if constexpr (OUT == OUT_PARTIAL)
          part[row * g.ldw + col + e] = v[e];
        else
          store_c<OUT == OUT_BF16>(g.C, row * g.ldc + col + e, v[e]);
      }
    }
  }
}

// ------------------------------------------------------ layout prologue
#if !AC_INPUT_F16
// The row-major copy of a column-major operand: dst (cols x rows, pitch
// ld_dst) = transpose of src (rows x cols, pitch ld_src). 64 x 64 tiles go
// through LDS: a thread reads runs of 8 elements of a source row with one
// 16-byte load (any 2-byte alignment; element loads at the end of a row),
// eight threads cover a 128-byte run of a row; a thread writes one 16-byte
// aligned run of 8 elements of a copy row (ld_dst is a multiple of 8 and dst
// is 16-byte aligned); elements past `rows` in the last run of a copy row
// are written as zero (the row pad). A grid-stride loop over the tiles.
constexpr int TR_T = 64;
__global__ __launch_bounds__(256) void k_transpose16(const uint16_t* __restrict__ src, int64_t ld_src,
                                                      uint16_t* __restrict__ dst, int64_t ld_dst, int64_t rows,
                                                      int64_t cols, int64_t tiles_c, int64_t tiles) {
  // rows of 66 elements (132 bytes): 4-byte aligned runs, and the column
  // reads of the write phase spread over the banks
  __shared__ uint32_t t32[TR_T * (TR_T + 2) / 2];
  const int tid = threadIdx.x;
  for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
    const int64_t r0 = (tile / tiles_c) * TR_T, c0 = (tile % tiles_c) * TR_T;
    __syncthreads();  // the previous tile's reads of t are done
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int e = tid + 256 * j;
      const int r = e >> 3, v8 = (e & 7) * 8;  // source row r0 + r, elements c0 + v8 .. + 7
      const int64_t gr = r0 + r, gc = c0 + v8;
      u32x4 w = {0u, 0u, 0u, 0u};
      if (gr < rows && gc < cols) {
        const uint16_t* p = src + gr * ld_src + gc;
        if (gc + 8 <= cols) {
          w = load16(p);
        } else {
#pragma unroll
          for (int x = 0; x < 8; ++x)
            if (gc + x < cols) w[x >> 1] |= (uint32_t)p[x] << (16 * (x & 1));
        }
      }
      uint32_t* d = t32 + (r * (TR_T + 2) + v8) / 2;
#pragma unroll
      for (int x = 0; x < 4; ++x) d[x] = w[x];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int e = tid + 256 * j;
      const int cc = e >> 3, q = e & 7;  // copy row c0 + cc, elements r0 + 8q .. r0 + 8q + 7
      const int64_t drow = c0 + cc, dcol = r0 + 8 * q;
      if (drow >= cols || dcol >= rows) continue;
      // element (row, cc) of the tile is half (cc & 1) of word (row * 66 + cc) / 2
      const int sh = 16 * (cc & 1);
      u32x4 w;
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const uint32_t lo = (t32[((8 * q + 2 * x) * (TR_T + 2) + cc) >> 1] >> sh) & 0xFFFFu;
        const uint32_t hi = (t32[((8 * q + 2 * x + 1) * (TR_T + 2) + cc) >> 1] >> sh) & 0xFFFFu;
        w[x] = lo | (hi << 16);
      }
      *reinterpret_cast<u32x4*>(dst + drow * ld_dst + dcol) = w;
    }
  }
}
#endif

#if AC_INPUT_F16
}  // namespace f16
#endif
}  // namespace ac

// ------------------------------------------------------------- registry
// VariantKey (family, config, output type) -> kernels; the launch boundary
// between the host planner and the device.
#include "planner.h"
#include "registry.h"

namespace ac {
#if AC_INPUT_F16
namespace f16 {
#endif

namespace {

typedef hipError_t (*LaunchFn)(const Plan&, const GemmArgs&, hipStream_t, bool);
typedef int (*OccFn)();

// Threads per output group of the reduction: enough threads in flight to
// cover the partial-slice read latency when the output is small.
int reduce_lg(int64_t outputs, int pk) {
  int lg = 0;
  while (lg < 6 && (2 << lg) <= pk && (outputs << lg) < (1 << 18)) ++lg;
  return lg;
}

hipError_t launch_reduce(const GemmArgs& g, hipStream_t st, bool obf) {
  const int64_t n = g.M * ((g.N + 7) / 8);
  const int lg = reduce_lg(n, g.pk);
  const int64_t eb = 256 >> lg;
  const dim3 grid((unsigned)((n + eb - 1) / eb)), block(256);
  if (obf)
    hipLaunchKernelGGL((k_reduce<true>), grid, block, 0, st, g, lg);
  else
    hipLaunchKernelGGL((k_reduce<false>), grid, block, 0, st, g, lg);
  return hipGetLastError();
}

// whole-K tiles with the AddMM epilogue
template <int BM, int BN, int MS, int D>
void launch_tile_addmm(dim3 grid, dim3 block, const GemmArgs& g, hipStream_t st, bool obf) {
  if (obf)
    hipLaunchKernelGGL((k_tile_addmm<BM, BN, MS, OUT_BF16, D>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_tile_addmm<BM, BN, MS, OUT_F32, D>), grid, block, 0, st, g);
}

template <int BM, int BN, int MS, int D>
hipError_t launch_tile(const Plan& p, const GemmArgs& g, hipStream_t st, bool obf) {
  const dim3 grid(p.grid_x, p.grid_y), block(TileShape<BM, BN, MS>::NT);
  if (p.pk > 1)
    hipLaunchKernelGGL((k_tile<BM, BN, MS, OUT_PARTIAL, D>), grid, block, 0, st, g);
  else if (g.epi)
    launch_tile_addmm<BM, BN, MS, D>(grid, block, g, st, obf);
  else if (obf)
    hipLaunchKernelGGL((k_tile<BM, BN, MS, OUT_BF16, D>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_tile<BM, BN, MS, OUT_F32, D>), grid, block, 0, st, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.pk == 1) return e;
  return launch_reduce(g, st, obf);
}
template <int BM, int BN, int MS>
hipError_t launch_streamk(const Plan& p, const GemmArgs& g, hipStream_t st, bool obf) {
  const dim3 grid(p.grid_x, 1), block(TileShape<BM, BN, MS>::NT), fblock(256);
  if (g.epi && obf)
    hipLaunchKernelGGL((k_streamk_addmm<BM, BN, MS, true>), grid, block, 0, st, g);
  else if (g.epi)
    hipLaunchKernelGGL((k_streamk_addmm<BM, BN, MS, false>), grid, block, 0, st, g);
  else if (obf)
    hipLaunchKernelGGL((k_streamk<BM, BN, MS, true>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_streamk<BM, BN, MS, false>), grid, block, 0, st, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || g.sk_tiles == 0) return e;
  const int chunks = (BM * (BN / 8) + 255) / 256;
  const dim3 fgrid(g.sk_tiles, chunks);
  if (obf)
    hipLaunchKernelGGL((k_sk_fixup<true>), fgrid, fblock, 0, st, g, BM, BN);
  else
    hipLaunchKernelGGL((k_sk_fixup<false>), fgrid, fblock, 0, st, g, BM, BN);
  return hipGetLastError();
}
template <int MT, int WKW>
hipError_t launch_skinny_m(const Plan& p, const GemmArgs& g, hipStream_t st, bool obf) {
  const dim3 grid(p.grid_x, p.grid_y), block(256);
  // a column-major B without a prologue copy is read in place
  const bool bt = (p.s.layouts & AC_LAYOUT_B_COL) && p.ws_b_off < 0;
  if (bt && obf)
    hipLaunchKernelGGL((k_skinny_m_bt<MT, WKW, true>), grid, block, 0, st, g);
  else if (bt)
    hipLaunchKernelGGL((k_skinny_m_bt<MT, WKW, false>), grid, block, 0, st, g);
  else if (obf)
    hipLaunchKernelGGL((k_skinny_m<MT, WKW, true>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_skinny_m<MT, WKW, false>), grid, block, 0, st, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.pk == 1) return e;
  return launch_reduce(g, st, obf);
}
template <int NT, int RB>
hipError_t launch_skinny_n(const Plan& p, const GemmArgs& g, hipStream_t st, bool obf) {
  const dim3 grid(p.grid_x, p.grid_y), block(256);
  if (obf)
    hipLaunchKernelGGL((k_skinny_n<NT, RB, true>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_skinny_n<NT, RB, false>), grid, block, 0, st, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.pk == 1) return e;
  return launch_reduce(g, st, obf);
}

template <int KMAX>
hipError_t launch_smallk(const Plan& p, const GemmArgs& g, hipStream_t st, bool obf) {
  const dim3 grid(p.grid_x, p.grid_y), block(256);
  if (p.tile_n == SMALLK_WIN_COLS) {
    // the windows must cover every column and the bands every row
    if ((int64_t)p.grid_x * SMALLK_WIN_COLS < g.N + 63 || (int64_t)p.grid_y * g.kper < g.M || g.kper > SMALLK_MAX_ROWS)
      return hipErrorInvalidValue;
    if (obf)
      hipLaunchKernelGGL((k_smallk_win<KMAX, true>), grid, block, 0, st, g);
    else
      hipLaunchKernelGGL((k_smallk_win<KMAX, false>), grid, block, 0, st, g);
  } else {
    if (obf)
      hipLaunchKernelGGL((k_smallk<KMAX, true>), grid, block, 0, st, g);
    else
      hipLaunchKernelGGL((k_smallk<KMAX, false>), grid, block, 0, st, g);
  }
  return hipGetLastError();
}

template <int WK>
hipError_t launch_direct(const Plan& p, const GemmArgs& g, hipStream_t st, bool obf) {
  const dim3 grid(p.grid_x, p.grid_y), block(WK == 1 ? 256 : 64 * WK);
  if (p.pk > 1)
    hipLaunchKernelGGL((k_direct<WK, OUT_PARTIAL>), grid, block, 0, st, g);
  else if (obf)
    hipLaunchKernelGGL((k_direct<WK, OUT_BF16>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_direct<WK, OUT_F32>), grid, block, 0, st, g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.pk == 1) return e;
  return launch_reduce(g, st, obf);
}

template <int BM, int BN, int MS>
hipError_t launch_persist(const Plan& p, const GemmArgs& g, hipStream_t st, bool obf) {
  // the buffer-store epilogue addresses a tile of C with 31-bit offsets
  if (g.ldc * (obf ? 2 : 4) >= (1LL << 23)) {
    static_assert(kTileCfg[0].depth == 1, "the persistent kernels are the depth-1 tile kernels");
    const dim3 grid(p.pm * p.pn), block(TileShape<BM, BN, MS>::NT);
    if (g.epi)
      launch_tile_addmm<BM, BN, MS, 1>(grid, block, g, st, obf);
    else if (obf)
      hipLaunchKernelGGL((k_tile<BM, BN, MS, OUT_BF16, 1>), grid, block, 0, st, g);
    else
      hipLaunchKernelGGL((k_tile<BM, BN, MS, OUT_F32, 1>), grid, block, 0, st, g);
    return hipGetLastError();
  }
  const dim3 grid(p.grid_x), block(TileShape<BM, BN, MS>::NT);
  if (g.epi && obf)
    hipLaunchKernelGGL((k_tile_pp_addmm<BM, BN, MS, true>), grid, block, 0, st, g);
  else if (g.epi)
    hipLaunchKernelGGL((k_tile_pp_addmm<BM, BN, MS, false>), grid, block, 0, st, g);
  else if (obf)
    hipLaunchKernelGGL((k_tile_pp<BM, BN, MS, true>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_tile_pp<BM, BN, MS, false>), grid, block, 0, st, g);
  return hipGetLastError();
}

template <int BM, int BN, int MS, int D>
hipError_t launch_grouped(const Plan& p, const GroupArgs& a, hipStream_t st, bool obf) {
  const dim3 grid(p.grid_x), block(TileShape<BM, BN, MS>::NT);
  if (a.g.epi && obf)
    hipLaunchKernelGGL((k_grouped_addmm<BM, BN, MS, OUT_BF16, D>), grid, block, 0, st, a);
  else if (a.g.epi)
    hipLaunchKernelGGL((k_grouped_addmm<BM, BN, MS, OUT_F32, D>), grid, block, 0, st, a);
  else if (obf)
    hipLaunchKernelGGL((k_grouped<BM, BN, MS, OUT_BF16, D>), grid, block, 0, st, a);
  else
    hipLaunchKernelGGL((k_grouped<BM, BN, MS, OUT_F32, D>), grid, block, 0, st, a);
  return hipGetLastError();
}
typedef hipError_t (*GroupLaunchFn)(const Plan&, const GroupArgs&, hipStream_t, bool);

template <typename F>
int occ_of(F kernel_f32, F kernel_bf16, int threads = 256) {
  int a = 0, b = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&a, reinterpret_cast<const void*>(kernel_f32), threads, 0) !=
      hipSuccess)
    a = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, reinterpret_cast<const void*>(kernel_bf16), threads, 0) !=
      hipSuccess)
    b = 0;
  return a < b ? a : b;
}
template <int BM, int BN, int MS, int D>
int occ_tile() {
  constexpr int nt = TileShape<BM, BN, MS>::NT;
  const int a = occ_of(k_tile<BM, BN, MS, OUT_F32, D>, k_tile<BM, BN, MS, OUT_BF16, D>, nt);
  const int b = occ_of(k_tile<BM, BN, MS, OUT_PARTIAL, D>, k_tile<BM, BN, MS, OUT_PARTIAL, D>, nt);
  return a < b ? a : b;
}
template <int BM, int BN, int MS>
int occ_persist() {
  return occ_of(k_tile_pp<BM, BN, MS, false>, k_tile_pp<BM, BN, MS, true>, TileShape<BM, BN, MS>::NT);
}
template <int BM, int BN, int MS, int D>
int occ_grouped() {
  return occ_of(k_grouped<BM, BN, MS, OUT_F32, D>, k_grouped<BM, BN, MS, OUT_BF16, D>, TileShape<BM, BN, MS>::NT);
}
template <int BM, int BN, int MS>
int occ_streamk() {
  return occ_of(k_streamk<BM, BN, MS, false>, k_streamk<BM, BN, MS, true>, TileShape<BM, BN, MS>::NT);
}
template <int MT, int WKW>
int occ_skinny_m() {
  return occ_of(k_skinny_m<MT, WKW, false>, k_skinny_m<MT, WKW, true>);
}
template <int NT, int RB>
int occ_skinny_n() {
  return occ_of(k_skinny_n<NT, RB, false>, k_skinny_n<NT, RB, true>);
}

// the entries of kTileCfg, in order: (bm, bn, ms, depth)
#define TILES(X)                                                                                               \
  X(256, 256, 32, 1), X(256, 128, 32, 1), X(128, 256, 32, 2), X(128, 128, 32, 1), X(128, 64, 32, 1),         \
      X(64, 128, 32, 1), X(64, 64, 32, 2), X(32, 32, 16, 2), X(128, 128, 32, 2), X(128, 64, 32, 2),           \
      X(64, 128, 32, 2)
#define L_TILE(a, b, c, d) &launch_tile<a, b, c, d>
#define O_TILE(a, b, c, d) &occ_tile<a, b, c, d>
const LaunchFn kTileFns[] = {TILES(L_TILE)};
const OccFn kTileOcc[] = {TILES(O_TILE)};
#define STREAMK_TILES(X)                                                                                       \
  X(256, 256, 32), X(256, 128, 32), X(128, 256, 32), X(128, 128, 32), X(128, 64, 32), X(64, 128, 32),        \
      X(64, 64, 32), X(32, 32, 16)
#define L_SK(a, b, c) &launch_streamk<a, b, c>
#define O_SK(a, b, c) &occ_streamk<a, b, c>
const LaunchFn kStreamKFns[] = {STREAMK_TILES(L_SK)};
const OccFn kStreamKOcc[] = {STREAMK_TILES(O_SK)};
const LaunchFn kSkinnyMFns[] = {&launch_skinny_m<1, 1>, &launch_skinny_m<1, 4>, &launch_skinny_m<2, 1>,
                                &launch_skinny_m<2, 4>, &launch_skinny_m<4, 1>, &launch_skinny_m<4, 4>};
const OccFn kSkinnyMOcc[] = {&occ_skinny_m<1, 1>, &occ_skinny_m<1, 4>, &occ_skinny_m<2, 1>,
                             &occ_skinny_m<2, 4>, &occ_skinny_m<4, 1>, &occ_skinny_m<4, 4>};
const LaunchFn kSkinnyNFns[] = {&launch_skinny_n<1, 2>, &launch_skinny_n<2, 2>, &launch_skinny_n<4, 2>};
const OccFn kSkinnyNOcc[] = {&occ_skinny_n<1, 2>, &occ_skinny_n<2, 2>, &occ_skinny_n<4, 2>};
template <int KMAX>
int occ_smallk() {
  const int a = occ_of(k_smallk<KMAX, false>, k_smallk<KMAX, true>);
  const int b = occ_of(k_smallk_win<KMAX, false>, k_smallk_win<KMAX, true>);
  return a < b ? a : b;
}
template <int WK>
int occ_direct() {
  constexpr int nt = WK == 1 ? 256 : 64 * WK;
  const int a = occ_of(k_direct<WK, OUT_F32>, k_direct<WK, OUT_BF16>, nt);
  const int b = occ_of(k_direct<WK, OUT_PARTIAL>, k_direct<WK, OUT_PARTIAL>, nt);
  return a < b ? a : b;
}

const LaunchFn kSmallKFns[] = {&launch_smallk<8>, &launch_smallk<16>};
const LaunchFn kDirectFns[] = {&launch_direct<1>, &launch_direct<4>, &launch_direct<16>};
const OccFn kDirectOcc[] = {&occ_direct<1>, &occ_direct<4>, &occ_direct<16>};
static_assert(sizeof(kDirectFns) / sizeof(kDirectFns[0]) == N_DIRECT_CFG, "direct table");
static_assert(kDirectCfg[0].wk == 1 && kDirectCfg[1].wk == 4 && kDirectCfg[2].wk == 16, "direct order");
const OccFn kSmallKOcc[] = {&occ_smallk<8>, &occ_smallk<16>};
static_assert(sizeof(kSmallKFns) / sizeof(kSmallKFns[0]) == N_SMALLK_CFG, "small-K table");
static_assert(kSmallKCfg[0].kmax == 8 && kSmallKCfg[1].kmax == 16, "small-K order");
static_assert(sizeof(kTileFns) / sizeof(kTileFns[0]) == N_TILE_CFG, "tile table");
static_assert(sizeof(kStreamKFns) / sizeof(kStreamKFns[0]) == N_STREAMK_CFG, "stream-K table");
#define CHK_TILE(a, b, c, d) {a, b, c, d}
constexpr int kTileCheck[][4] = {TILES(CHK_TILE)};
constexpr bool tiles_match() {
  for (int i = 0; i < N_TILE_CFG; ++i)
    if (kTileCheck[i][0] != kTileCfg[i].bm || kTileCheck[i][1] != kTileCfg[i].bn ||
        kTileCheck[i][2] != kTileCfg[i].ms || kTileCheck[i][3] != kTileCfg[i].depth)
      return false;
  return true;
}
static_assert(tiles_match(), "tile kernels must follow kTileCfg");
constexpr bool dl_siblings_match() {
  for (int i = 0; i < N_DL_CFG; ++i) {
    if (kDlCfg[i].sibling < 0) {
      if (!kDlCfg[i].unal) return false;  // some fallback must exist
      continue;
    }
    const TileCfg& t = kTileCfg[kDlCfg[i].sibling];
    if (t.bm != kDlCfg[i].bm || t.bn != kDlCfg[i].bn || t.ms != 32) return false;
  }
  return true;
}
static_assert(dl_siblings_match(), "a direct-to-LDS configuration falls back to the tile kernel of its tiling");
static_assert(sizeof(kSkinnyMFns) / sizeof(kSkinnyMFns[0]) == N_SKINNY_M_CFG, "skinny-M table");
static_assert(sizeof(kSkinnyNFns) / sizeof(kSkinnyNFns[0]) == N_SKINNY_N_CFG, "skinny-N table");

// The tables above must list the configurations in the order of variants.h
// (the tile kernels are checked by tiles_match).
constexpr bool streamk_order_ok() {
  const int e[][3] = {{256, 256, 32}, {256, 128, 32}, {128, 256, 32}, {128, 128, 32},
                      {128, 64, 32},  {64, 128, 32},  {64, 64, 32},   {32, 32, 16}};
  for (int i = 0; i < N_STREAMK_CFG; ++i)
    if (kTileCfg[i].bm != e[i][0] || kTileCfg[i].bn != e[i][1] || kTileCfg[i].ms != e[i][2]) return false;
  return true;
}
static_assert(streamk_order_ok(), "stream-K configuration order");
static_assert(kSkinnyMCfg[0].mt == 1 && kSkinnyMCfg[1].wkw == 4 && kSkinnyMCfg[4].mt == 4, "skinny-M order");
static_assert(kSkinnyNCfg[0].nt == 1 && kSkinnyNCfg[2].nt == 4 && kSkinnyNCfg[0].rb == 2, "skinny-N order");
static_assert(SKINNY_N_KMAX == SKN_KMAX, "skinny-N LDS slice");

// Grouped kernels of the configurations kGroupedCfg enables (null otherwise).
template <int I>
constexpr GroupLaunchFn grouped_fn() {
  constexpr TileCfg t = kTileCfg[I];
  if constexpr (kGroupedCfg[I])
    return &launch_grouped<t.bm, t.bn, t.ms, t.depth>;
  else
    return nullptr;
}
template <int I>
constexpr OccFn grouped_occ() {
  constexpr TileCfg t = kTileCfg[I];
  if constexpr (kGroupedCfg[I])
    return &occ_grouped<t.bm, t.bn, t.ms, t.depth>;
  else
    return nullptr;
}
template <int I>
constexpr LaunchFn persist_fn() {
  constexpr TileCfg t = kTileCfg[I];
  if constexpr (kPersistCfg[I])
    return &launch_persist<t.bm, t.bn, t.ms>;
  else
    return nullptr;
}
template <int I>
constexpr OccFn persist_occ() {
  constexpr TileCfg t = kTileCfg[I];
  if constexpr (kPersistCfg[I])
    return &occ_persist<t.bm, t.bn, t.ms>;
  else
    return nullptr;
}
static_assert(N_TILE_CFG == 11, "grouped and persistent tables list every tile configuration");
const LaunchFn kPersistFns[] = {persist_fn<0>(), persist_fn<1>(), persist_fn<2>(), persist_fn<3>(),
                                persist_fn<4>(), persist_fn<5>(), persist_fn<6>(), persist_fn<7>(),
                                persist_fn<8>(), persist_fn<9>(), persist_fn<10>()};
const OccFn kPersistOcc[] = {persist_occ<0>(), persist_occ<1>(), persist_occ<2>(), persist_occ<3>(),
                             persist_occ<4>(), persist_occ<5>(), persist_occ<6>(), persist_occ<7>(),
                             persist_occ<8>(), persist_occ<9>(), persist_occ<10>()};
const GroupLaunchFn kGroupedFns[] = {grouped_fn<0>(), grouped_fn<1>(), grouped_fn<2>(), grouped_fn<3>(),
                                     grouped_fn<4>(), grouped_fn<5>(), grouped_fn<6>(), grouped_fn<7>(),
                                     grouped_fn<8>(), grouped_fn<9>(), grouped_fn<10>()};
const OccFn kGroupedOcc[] = {grouped_occ<0>(), grouped_occ<1>(), grouped_occ<2>(), grouped_occ<3>(),
                             grouped_occ<4>(), grouped_occ<5>(), grouped_occ<6>(), grouped_occ<7>(),
                             grouped_occ<8>(), grouped_occ<9>(), grouped_occ<10>()};

}  // namespace

hipError_t launch_plan(const Plan& p, const GemmArgs& g, hipStream_t st) {
  const bool obf = dtype_out16(p.s.dtype);
  switch (p.family) {
    case FAM_TILE:
      return kTileFns[p.cfg](p, g, st, obf);
    case FAM_STREAMK:
      return kStreamKFns[p.cfg](p, g, st, obf);
    case FAM_SKINNY_M:
      return kSkinnyMFns[p.cfg](p, g, st, obf);
    case FAM_SKINNY_N:
      return kSkinnyNFns[p.cfg](p, g, st, obf);
    case FAM_SMALLK:
      return kSmallKFns[p.cfg](p, g, st, obf);
    case FAM_DIRECT:
      return kDirectFns[p.cfg](p, g, st, obf);
    case FAM_PERSIST:
      if (p.cfg < 0 || p.cfg >= N_TILE_CFG || !kPersistFns[p.cfg] || g.K < 8 || g.N < 8) return hipErrorInvalidValue;
      return kPersistFns[p.cfg](p, g, st, obf);
    case FAM_DL: {
      if (p.cfg < 0 || p.cfg >= N_DL_CFG) return hipErrorInvalidValue;
      // launch_dl_main checks the operands against the plan's form: aligned
      // rows for the direct loads (the caller runs the register-staged
      // sibling otherwise), any alignment for the register-load form
      const hipError_t e = (launch_dl_main)(p, g, st);  // this format's kernels (no argument-dependent lookup)
      if (e != hipSuccess || p.pk == 1) return e;
      return launch_reduce(g, st, obf);
    }
    case FAM_TALL: {
      // g.B / g.ldb: the transposed copy of B the caller's prologue wrote
      const hipError_t e = (launch_tall_main)(p, g, st);
      if (e != hipSuccess || p.pk == 1) return e;
      return launch_reduce(g, st, obf);
    }
    case FAM_DLSC: {
      // every slice's partials, then the reduction over the slices
      const hipError_t e = (launch_dl_sc_main)(p, g, st);
      if (e != hipSuccess) return e;
      return launch_reduce(g, st, obf);
    }
  }
  return hipErrorInvalidValue;
}

hipError_t launch_grouped_plan(const Plan& p, const GroupArgs& a, hipStream_t st) {
  if ((p.family != FAM_GROUPED && p.family != FAM_BATCHED) || p.cfg < 0 || p.cfg >= N_TILE_CFG ||
      !kGroupedFns[p.cfg])
    return hipErrorInvalidValue;
  return kGroupedFns[p.cfg](p, a, st, dtype_out16(p.s.dtype));
}

#if !AC_INPUT_F16
// Measurement reference: every 16-byte word of the buffer read once with
// non-temporal 16-byte loads, 8 in flight per thread, over a grid of two
// workgroups per CU; a value is stored only if the XOR of everything read
// equals a constant no data here produces, so the loads are not elided.
__global__ __launch_bounds__(256) void k_read_probe(const u32x4* __restrict__ p, int64_t n, uint32_t* sink) {
  const int64_t nt = (int64_t)gridDim.x * 256;
  u32x4 acc = {0u, 0u, 0u, 0u};
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + 7 * nt < n; i += 8 * nt) {
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(p + i + u * nt);
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= v[u];
  }
  for (; i < n; i += nt) acc ^= p[i];
  const uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  if (x == 0x9E3779B9u) sink[0] = x;
}

hipError_t launch_read_probe(const void* buf, int64_t bytes, void* sink, hipStream_t st) {
  if (bytes <= 0) return hipSuccess;
  if (((uintptr_t)buf & 15) != 0 || (bytes & 15) != 0 || ((uintptr_t)sink & 3) != 0) return hipErrorInvalidValue;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                               hipSuccess)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_read_probe, dim3(2 * cus), dim3(256), 0, st, static_cast<const u32x4*>(buf), bytes / 16,
                     static_cast<uint32_t*>(sink));
  return hipGetLastError();
}

hipError_t launch_transpose16(const uint16_t* src, int64_t ld_src, int64_t rows, int64_t cols, uint16_t* dst,
                              int64_t ld_dst, hipStream_t st) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  if (ld_src < cols || ld_dst < rows || (ld_dst & 7) != 0 || ((uintptr_t)dst & 15) != 0) return hipErrorInvalidValue;
  const int64_t tiles_c = (cols + TR_T - 1) / TR_T;
  const int64_t tiles = (rows + TR_T - 1) / TR_T * tiles_c;
  const dim3 grid((unsigned)(tiles < 4096 ? tiles : 4096)), block(256);
  hipLaunchKernelGGL(k_transpose16, grid, block, 0, st, src, ld_src, dst, ld_dst, rows, cols, tiles_c, tiles);
  return hipGetLastError();
}
#endif

void query_occupancy() {
  for (int i = 0; i < N_TILE_CFG; ++i) set_runtime_occupancy(FAM_TILE, i, kTileOcc[i]());
  for (int i = 0; i < N_STREAMK_CFG; ++i) set_runtime_occupancy(FAM_STREAMK, i, kStreamKOcc[i]());
  for (int i = 0; i < N_SKINNY_M_CFG; ++i) set_runtime_occupancy(FAM_SKINNY_M, i, kSkinnyMOcc[i]());
  for (int i = 0; i < N_SKINNY_N_CFG; ++i) set_runtime_occupancy(FAM_SKINNY_N, i, kSkinnyNOcc[i]());
  for (int i = 0; i < N_SMALLK_CFG; ++i) set_runtime_occupancy(FAM_SMALLK, i, kSmallKOcc[i]());
  for (int i = 0; i < N_DIRECT_CFG; ++i) set_runtime_occupancy(FAM_DIRECT, i, kDirectOcc[i]());
  for (int i = 0; i < N_TILE_CFG; ++i)
    if (kGroupedOcc[i]) set_runtime_occupancy(FAM_GROUPED, i, kGroupedOcc[i]());
  for (int i = 0; i < N_TILE_CFG; ++i)
    if (kPersistOcc[i]) set_runtime_occupancy(FAM_PERSIST, i, kPersistOcc[i]());
  query_occupancy_dl();
  query_occupancy_tall();
}

#if AC_INPUT_F16
}  // namespace f16
#endif
}  // namespace ac
