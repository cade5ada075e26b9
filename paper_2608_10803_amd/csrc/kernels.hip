// gfx950 GEMM kernels: C = A * B with bf16 inputs, fp32 accumulation and
// fp32 or bf16 output (RNE), for any M, N, K, leading dimensions and 2-byte
// aligned pointers.
//
//   k_tile      MFMA macro-tile kernel with LDS double buffering. One launch
//               per template: P_k == 1 is the Common template (k = K, one
//               cast and one write per output, Eq. 2); P_k > 1 the
//               MultiCoreSplitK template (K split across workgroups, fp32
//               partials, cross-workgroup reduction, Eq. 4 / Eq. 11).
//   k_streamk   StreamK applied to the tile kernel (Section 4.2): a
//               persistent grid splits the MAC iterations of the last tiles
//               evenly; partial tiles are fixed up in a fixed order.
//   k_skinny_m  Small-M Copy module (Table 2) for M <= 64: B is streamed from
//               HBM exactly once, A stays in cache; split K across CUs.
//   k_skinny_n  the same module for N <= 64: A streamed once, the small B is
//               kept resident in LDS (L1 Resident module, Table 2).
//
// Cross-workgroup reductions are deterministic: the last workgroup to arrive
// at a tile sums the fp32 partials in partition order 0, 1, ..., P_k - 1, so
// a result does not depend on arrival order, and resets the tile's counter
// to zero for the next launch.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernel_args.h"

namespace ac {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// ---------------------------------------------------------------- helpers

// 16-byte load from a 2-byte aligned address. gfx950 runs in unaligned
// access mode, and the compiler emits one dwordx4 load for this copy.
__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  u32x4 v;
  __builtin_memcpy(&v, p, 16);
  return v;
}

// The first `valid` (1..7) elements of a 16-byte vector, zeros after.
__device__ __forceinline__ u32x4 load16_part(const uint16_t* p, int valid) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t lo = (2 * i < valid) ? (uint32_t)p[2 * i] : 0u;
    uint32_t hi = (2 * i + 1 < valid) ? (uint32_t)p[2 * i + 1] : 0u;
    w[i] = lo | (hi << 16);
  }
  return u32x4{w[0], w[1], w[2], w[3]};
}

// Eight consecutive elements p[0..7], of which `valid` exist.
__device__ __forceinline__ u32x4 load16_guard(const uint16_t* p, int64_t valid) {
  if (valid >= 8) return load16(p);
  if (valid <= 0) return u32x4{0u, 0u, 0u, 0u};
  return load16_part(p, (int)valid);
}

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

__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ uint16_t to_bf16(float f) {
  __bf16 h = (__bf16)f;  // round to nearest even; NaN stays NaN
  return __builtin_bit_cast(uint16_t, h);
}

template <bool OBF>
__device__ __forceinline__ void store_c(void* C, int64_t idx, float v) {
  if constexpr (OBF)
    static_cast<uint16_t*>(C)[idx] = to_bf16(v);
  else
    static_cast<float*>(C)[idx] = v;
}

// Eight consecutive outputs of one row; `valid` of them exist.
template <bool OBF>
__device__ __forceinline__ void store_c8(void* C, int64_t idx, const float (&v)[8], int64_t valid) {
  if constexpr (OBF) {
    uint16_t* p = static_cast<uint16_t*>(C) + idx;
    if (valid >= 8) {
      u32x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = (uint32_t)to_bf16(v[2 * e]) | ((uint32_t)to_bf16(v[2 * e + 1]) << 16);
      __builtin_memcpy(p, &w, 16);
    } else {
      for (int j = 0; j < valid; ++j) p[j] = to_bf16(v[j]);
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

// LDS rows are 16-byte chunks; the chunk index is XORed with low row bits so
// that the 16 lanes reading 16 consecutive rows at one chunk hit distinct banks.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row & 7) ^ ((row >> 3) & 1)); }

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own L2):
// give every XCD a contiguous range of tile ids, so neighbouring tiles share an L2.
__device__ __forceinline__ int xcd_remap(int b, int n) {
  const int q = n >> 3, r = n & 7, x = b & 7, i = b >> 3;
  return x * q + min(x, r) + i;
}

// Tile id -> (tile_m, tile_n). Grouped order: 8 tile rows per group, column
// by column inside a group, so consecutive ids reuse A rows and B columns.
__device__ __forceinline__ void tile_coords(int t, int tiles_m, int tiles_n, int grouped, int& tm, int& tn) {
  if (!grouped) {
    tm = t / tiles_n;
    tn = t - tm * tiles_n;
    return;
  }
  const int G = 8;
  const int per_group = G * tiles_n;
  const int grp = t / per_group;
  const int first = grp * G;
  const int gsz = min(tiles_m - first, G);
  const int in = t - grp * per_group;
  tm = first + in % gsz;
  tn = in / gsz;
}

// Last-arrival protocol of the deterministic cross-workgroup reduction.
// Every thread has stored its partial; returns true in the workgroup that
// arrived last, after which all partials of the tile are visible to it.
__device__ __forceinline__ bool arrive_last(int* counter, int expected, int* s_flag) {
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    const int old = atomicAdd(counter, 1);
    const int last = (old == expected - 1);
    if (last) {
      __threadfence();
      // every other workgroup of the tile has arrived: reset for the next launch
      __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    *s_flag = last;
  }
  __syncthreads();
  const bool last = *s_flag != 0;
  if (last) __threadfence();
  return last;
}

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

template <int BM, int BN, int MS>
struct TileShape {
  static constexpr int NT = 256, BK = 64, CH = 8;
  static constexpr int WTM = BM / 2, WTN = BN / 2;
  static constexpr int TM = WTM / MS, TN = WTN / MS;
  static constexpr int KS = MS == 32 ? 16 : 32;
  static constexpr int NA = AccOf<MS>::n;
  static constexpr int NACC = TM * TN * NA;  // accumulator floats per thread
  static constexpr int AV = BM * CH;          // 16-byte vectors of an A stage
  static constexpr int IA = (AV + NT - 1) / NT;
  static constexpr int IB = (BN + NT - 1) / NT;  // 8x8 blocks of a B stage (BK/8 * BN/8 = BN)
  static_assert(WTM % MS == 0 && WTN % MS == 0, "wave tile must be a multiple of the MFMA tile");
};

// Computes the tile's accumulators over k-blocks [kt0, kt1).
template <int BM, int BN, int MS>
__device__ __forceinline__ void tile_mainloop(const GemmArgs& g, int64_t m0, int64_t n0, int kt0, int kt1,
                                              typename AccOf<MS>::T (&acc)[TileShape<BM, BN, MS>::TM]
                                                                         [TileShape<BM, BN, MS>::TN],
                                              u32x4 (*sA)[BM * 8], u32x4 (*sB)[BN * 8]) {
  typedef TileShape<BM, BN, MS> S;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;
  const uint16_t* __restrict__ A = g.A;
  const uint16_t* __restrict__ B = g.B;
  const int64_t M = g.M, N = g.N, K = g.K, lda = g.lda, ldb = g.ldb;

  u32x4 ra[S::IA];
  u32x4 rb[S::IB][8];

  auto load_stage = [&](int kt) {
    const int64_t kbase = (int64_t)kt * S::BK;
#pragma unroll
    for (int i = 0; i < S::IA; ++i) {
      const int idx = tid + i * S::NT;
      if (S::AV % S::NT == 0 || idx < S::AV) {
        const int row = idx >> 3, c = idx & 7;
        const int64_t gr = m0 + row, gk = kbase + c * 8;
        ra[i] = gr < M ? load16_guard(A + gr * lda + gk, K - gk) : u32x4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int b = 0; b < S::IB; ++b) {
      const int blk = tid + b * S::NT;
      if (BN % S::NT == 0 || blk < BN) {
        const int c = blk & 7, grp = blk >> 3;
        const int64_t gn = n0 + grp * 8;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int64_t gk = kbase + c * 8 + i;
          rb[b][i] = gk < K ? load16_guard(B + gk * ldb + gn, N - gn) : u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int i = 0; i < S::IA; ++i) {
      const int idx = tid + i * S::NT;
      if (S::AV % S::NT == 0 || idx < S::AV) {
        const int row = idx >> 3, c = idx & 7;
        sA[buf][row * 8 + swz(row, c)] = ra[i];
      }
    }
#pragma unroll
    for (int b = 0; b < S::IB; ++b) {
      const int blk = tid + b * S::NT;
      if (BN % S::NT == 0 || blk < BN) {
        const int c = blk & 7, grp = blk >> 3;
        u32x4 col[8];
        transpose8x8(rb[b], col);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int n = grp * 8 + j;
          sB[buf][n * 8 + swz(n, c)] = col[j];
        }
      }
    }
  };
  auto compute = [&](int buf) {
#pragma unroll
    for (int ks = 0; ks < S::BK / S::KS; ++ks) {
      const int chunk = MS == 32 ? ks * 2 + (lane >> 5) : ks * 4 + (lane >> 4);
      u32x4 fa[S::TM], fb[S::TN];
#pragma unroll
      for (int i = 0; i < S::TM; ++i) {
        const int row = wr * S::WTM + i * MS + (lane % MS);
        fa[i] = sA[buf][row * 8 + swz(row, chunk)];
      }
#pragma unroll
      for (int j = 0; j < S::TN; ++j) {
        const int col = wc * S::WTN + j * MS + (lane % MS);
        fb[j] = sB[buf][col * 8 + swz(col, chunk)];
      }
#pragma unroll
      for (int i = 0; i < S::TM; ++i)
#pragma unroll
        for (int j = 0; j < S::TN; ++j) {
          if constexpr (MS == 32)
            acc[i][j] = mfma32(fa[i], fb[j], acc[i][j]);
          else
            acc[i][j] = mfma16(fa[i], fb[j], acc[i][j]);
        }
    }
  };

  if (kt0 >= kt1) return;
  load_stage(kt0);
  store_stage(0);
  __syncthreads();
  for (int kt = kt0; kt < kt1; ++kt) {
    const int buf = (kt - kt0) & 1;
    const bool more = kt + 1 < kt1;
    if (more) load_stage(kt + 1);
    compute(buf);
    if (more) store_stage(buf ^ 1);
    __syncthreads();
  }
}

// Row (within the MFMA block) of accumulator element r of this lane.
template <int MS>
__device__ __forceinline__ int acc_row(int r, int lane) {
  if constexpr (MS == 32)
    return (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
  else
    return (lane >> 4) * 4 + r;
}

// Stores accumulator element q (flattened (i, j, r)) of this thread to C.
template <int BM, int BN, int MS, bool OBF>
__device__ __forceinline__ void store_acc_elem(const GemmArgs& g, int64_t m0, int64_t n0, int q, float v) {
  typedef TileShape<BM, BN, MS> S;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;
  const int r = q % S::NA, ij = q / S::NA, i = ij / S::TN, j = ij % S::TN;
  const int64_t row = m0 + wr * S::WTM + i * MS + acc_row<MS>(r, lane);
  const int64_t col = n0 + wc * S::WTN + j * MS + (lane % MS);
  if (row < g.M && col < g.N) store_c<OBF>(g.C, row * g.ldc + col, v);
}

template <int BM, int BN, int MS, bool OBF>
__global__ __launch_bounds__(256) void k_tile(GemmArgs g) {
  typedef TileShape<BM, BN, MS> S;
  typedef typename AccOf<MS>::T Acc;
  __shared__ u32x4 sA[2][BM * 8];
  __shared__ u32x4 sB[2][BN * 8];
  __shared__ int s_flag;

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

  tile_mainloop<BM, BN, MS>(g, m0, n0, kt0, kt1, acc, sA, sB);

  if (g.pk == 1) {
#pragma unroll
    for (int i = 0; i < S::TM; ++i)
#pragma unroll
      for (int j = 0; j < S::TN; ++j)
#pragma unroll
        for (int r = 0; r < S::NA; ++r) store_acc_elem<BM, BN, MS, OBF>(g, m0, n0, (i * S::TN + j) * S::NA + r, acc[i][j][r]);
    return;
  }

  // Split K: publish this partition's fp32 tile, the last arrival reduces.
  const int tid = threadIdx.x;
  const size_t tile_floats = (size_t)BM * BN;
  float* wtile = g.ws + (size_t)tile * g.pk * tile_floats;
  {
    float* mine = wtile + (size_t)split * tile_floats;
#pragma unroll
    for (int i = 0; i < S::TM; ++i)
#pragma unroll
      for (int j = 0; j < S::TN; ++j)
#pragma unroll
        for (int r4 = 0; r4 < S::NA / 4; ++r4) {
          const int c4 = (i * S::TN + j) * (S::NA / 4) + r4;
          f32x4 v = {acc[i][j][r4 * 4], acc[i][j][r4 * 4 + 1], acc[i][j][r4 * 4 + 2], acc[i][j][r4 * 4 + 3]};
          *reinterpret_cast<f32x4*>(mine + ((size_t)c4 * S::NT + tid) * 4) = v;
        }
  }
  if (!arrive_last(g.counters + tile, g.pk, &s_flag)) return;
#pragma unroll
  for (int c4 = 0; c4 < S::NACC / 4; ++c4) {
    f32x4 s = *reinterpret_cast<const f32x4*>(wtile + ((size_t)c4 * S::NT + tid) * 4);
    for (int p = 1; p < g.pk; ++p) s += *reinterpret_cast<const f32x4*>(wtile + p * tile_floats + ((size_t)c4 * S::NT + tid) * 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) store_acc_elem<BM, BN, MS, OBF>(g, m0, n0, c4 * 4 + e, s[e]);
  }
}

// --------------------------------------------------------- stream-K kernel
// A persistent grid of G workgroups. The first `sk_tiles` tiles (in tile id
// order) are split into MAC iterations (one k-block each) and every
// workgroup takes `iters_per_wg` consecutive iterations; a tile's pieces are
// written as fp32 partials and the workgroup holding the tile's first
// iteration sums them in iteration order once the others have arrived (it
// processes that piece last, so its peers started earlier). The remaining
// tiles are processed whole, data-parallel, by the grid afterwards.
template <int BM, int BN, int MS, bool OBF>
__global__ __launch_bounds__(256) void k_streamk(GemmArgs g) {
  typedef TileShape<BM, BN, MS> S;
  typedef typename AccOf<MS>::T Acc;
  __shared__ u32x4 sA[2][BM * 8];
  __shared__ u32x4 sB[2][BN * 8];
   const int tid = threadIdx.x;
  const int ntiles = g.tiles_m * g.tiles_n;
  const int ipt = (int)((g.K + S::BK - 1) / S::BK);  // iterations per tile
  const int G = gridDim.x;
  const size_t tile_floats = (size_t)BM * BN;
  const int64_t total_sk = (int64_t)g.sk_tiles * ipt;

  // Stream-K phase.
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
    tile_mainloop<BM, BN, MS>(g, m0, n0, k_begin, k_end, acc, sA, sB);
    __syncthreads();

    // Workgroups covering this tile: their first iterations are multiples of
    // iters_per_wg; the owner holds k_begin == 0.
    const int64_t t0 = (int64_t)tile * ipt;
    const int first_wg = (int)(t0 / g.iters_per_wg);
    const int last_wg = (int)min((int64_t)G - 1, (t0 + ipt - 1) / g.iters_per_wg);
    const int slot = blockIdx.x - first_wg;  // piece index within the tile
    const int pieces = last_wg - first_wg + 1;
    float* wtile = g.ws + (size_t)tile * (size_t)g.pk * tile_floats;

    if (pieces == 1) {
#pragma unroll
      for (int i = 0; i < S::TM; ++i)
#pragma unroll
        for (int j = 0; j < S::TN; ++j)
#pragma unroll
          for (int r = 0; r < S::NA; ++r)
            store_acc_elem<BM, BN, MS, OBF>(g, m0, n0, (i * S::TN + j) * S::NA + r, acc[i][j][r]);
    } else if (k_begin != 0) {
      // Non-owner: publish the partial and raise this piece's flag.
      float* mine = wtile + (size_t)slot * tile_floats;
#pragma unroll
      for (int i = 0; i < S::TM; ++i)
#pragma unroll
        for (int j = 0; j < S::TN; ++j)
#pragma unroll
          for (int r4 = 0; r4 < S::NA / 4; ++r4) {
            const int c4 = (i * S::TN + j) * (S::NA / 4) + r4;
            f32x4 v = {acc[i][j][r4 * 4], acc[i][j][r4 * 4 + 1], acc[i][j][r4 * 4 + 2], acc[i][j][r4 * 4 + 3]};
            *reinterpret_cast<f32x4*>(mine + ((size_t)c4 * S::NT + tid) * 4) = v;
          }
      __threadfence();
      __syncthreads();
      if (tid == 0) atomicAdd(g.counters + tile, 1);
    } else {
      // Owner: wait (bounded) for the other pieces, then sum in piece order.
      if (tid == 0) {
        int spins = 0;
        while (__hip_atomic_load(g.counters + tile, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < pieces - 1) {
          __builtin_amdgcn_s_sleep(2);
          if (++spins > g.spin_limit) {
            atomicExch(g.err_flag, 1);
            break;
          }
        }
        __hip_atomic_store(g.counters + tile, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      __syncthreads();
      __threadfence();
#pragma unroll
      for (int i = 0; i < S::TM; ++i)
#pragma unroll
        for (int j = 0; j < S::TN; ++j)
#pragma unroll
          for (int r4 = 0; r4 < S::NA / 4; ++r4) {
            const int c4 = (i * S::TN + j) * (S::NA / 4) + r4;
            f32x4 s = {acc[i][j][r4 * 4], acc[i][j][r4 * 4 + 1], acc[i][j][r4 * 4 + 2], acc[i][j][r4 * 4 + 3]};
            for (int p = 1; p < pieces; ++p)
              s += *reinterpret_cast<const f32x4*>(wtile + p * tile_floats + ((size_t)c4 * S::NT + tid) * 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) store_acc_elem<BM, BN, MS, OBF>(g, m0, n0, c4 * 4 + e, s[e]);
          }
    }
    it += k_end - k_begin;
  }

  // Data-parallel phase: whole tiles after the stream-K ones.
  for (int tile = g.sk_tiles + blockIdx.x; tile < ntiles; tile += G) {
    int tm, tn;
    tile_coords(tile, g.tiles_m, g.tiles_n, g.swizzle, tm, tn);
    const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
    Acc acc[S::TM][S::TN];
#pragma unroll
    for (int i = 0; i < S::TM; ++i)
#pragma unroll
      for (int j = 0; j < S::TN; ++j) acc[i][j] = Acc{};
    __syncthreads();
    tile_mainloop<BM, BN, MS>(g, m0, n0, 0, ipt, acc, sA, sB);
#pragma unroll
    for (int i = 0; i < S::TM; ++i)
#pragma unroll
      for (int j = 0; j < S::TN; ++j)
#pragma unroll
        for (int r = 0; r < S::NA; ++r)
          store_acc_elem<BM, BN, MS, OBF>(g, m0, n0, (i * S::TN + j) * S::NA + r, acc[i][j][r]);
  }
}

// -------------------------------------------------------- skinny-M kernel
// C (M x N, M <= 16*MT) = A * B with B streamed once. A wave owns 128
// columns: lane l loads, for k-group l/16, an 8 x 8 block (8 k-rows, 8
// columns starting at 8*(l%16)), transposes it in registers and issues one
// 16x16x32 MFMA per column j, so MFMA j computes the 16 columns
// {base + 8c + j}. A fragments (16 rows x 32 k) come straight from global
// memory (A is small and stays in cache). WKW waves of a workgroup split the
// workgroup's k-range and are reduced through LDS in wave order.
template <int MT, int WKW, bool OBF>
__global__ __launch_bounds__(256) void k_skinny_m(GemmArgs g) {
  constexpr int WNW = 4 / WKW;
  constexpr int NB = 128 * WNW;
  constexpr int U = 2;
  constexpr int NV = MT * 8;  // f32x4 accumulators per lane
  __shared__ f32x4 red[WKW > 1 ? (WKW - 1) * WNW * NV * 64 : 1];
  __shared__ int s_flag;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wc = wave % WNW, wk = wave / WNW;
  const int cb = blockIdx.x, split = blockIdx.y;
  const int64_t M = g.M, N = g.N, K = g.K, lda = g.lda, ldb = g.ldb;
  const int64_t col0 = (int64_t)cb * NB + wc * 128 + 8 * (lane & 15);
  const int kg = lane >> 4;
  const int kb_total = (int)((K + 31) / 32);
  const int kb0 = min(split * g.kper, kb_total);
  const int kb1 = min(kb0 + g.kper, kb_total);

  f32x4 acc[MT][8];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[mt][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t nvalid = N - col0;
  for (int kb = kb0 + wk; kb < kb1; kb += WKW * U) {
    u32x4 rb[U][8];
    u32x4 fa[U][MT];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kbu = kb + u * WKW;
      const int64_t k = (int64_t)kbu * 32 + kg * 8;
      const bool on = kbu < kb1;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        rb[u][i] = (on && k + i < K && nvalid > 0) ? load16_guard(g.B + (k + i) * ldb + col0, nvalid)
                                                   : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int64_t row = mt * 16 + (lane & 15);
        fa[u][mt] = (on && row < M) ? load16_guard(g.A + row * lda + k, K - k) : u32x4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      u32x4 col[8];
      transpose8x8(rb[u], col);
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
    if (wk == 0) {
      for (int w = 1; w < WKW; ++w)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int j = 0; j < 8; ++j) acc[mt][j] += red[(((w - 1) * WNW + wc) * NV + mt * 8 + j) * 64 + lane];
    }
  }

  // Output: lane holds rows mt*16 + 4*(l/16) + r, columns col0 .. col0+7.
  auto store_out = [&](const f32x4 (&v)[MT][8]) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = mt * 16 + (lane >> 4) * 4 + r;
        if (row < M && nvalid > 0) {
          float o[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) o[j] = v[mt][j][r];
          store_c8<OBF>(g.C, row * g.ldc + col0, o, nvalid);
        }
      }
  };

  if (g.pk == 1) {
    if (wk == 0) store_out(acc);
    return;
  }
  const size_t blk_floats = (size_t)WNW * NV * 64 * 4;
  float* wblk = g.ws + (size_t)cb * g.pk * blk_floats;
  if (wk == 0) {
    float* mine = wblk + (size_t)split * blk_floats;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        *reinterpret_cast<f32x4*>(mine + (((size_t)wc * NV + mt * 8 + j) * 64 + lane) * 4) = acc[mt][j];
  }
  if (!arrive_last(g.counters + cb, g.pk, &s_flag)) return;
  if (wk != 0) return;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const size_t off = (((size_t)wc * NV + mt * 8 + j) * 64 + lane) * 4;
      f32x4 s = *reinterpret_cast<const f32x4*>(wblk + off);
      for (int p = 1; p < g.pk; ++p) s += *reinterpret_cast<const f32x4*>(wblk + p * blk_floats + off);
      acc[mt][j] = s;
    }
  store_out(acc);
}

// -------------------------------------------------------- skinny-N kernel
// C (M x N, N <= 16*NT) = A * B with A streamed once. The workgroup's k-range
// of B (at most SKN_KMAX) is transposed into LDS once; each wave then streams
// 16*RB rows of A, one 16-byte fragment per lane per 32-k block, and issues
// RB*NT 16x16x32 MFMAs against the resident B fragments.
constexpr int SKN_KMAX = 512;

template <int NT, int RB, bool OBF>
__global__ __launch_bounds__(256) void k_skinny_n(GemmArgs g) {
  constexpr int NCOL = NT * 16;
  constexpr int KCH = SKN_KMAX / 8;  // 16-byte chunks per LDS row
  constexpr int U = 2;
  __shared__ u32x4 sBt[NCOL * KCH];
  __shared__ int s_flag;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rbk = blockIdx.x, split = blockIdx.y;
  const int64_t M = g.M, N = g.N, K = g.K, lda = g.lda, ldb = g.ldb;
  const int kb_total = (int)((K + 31) / 32);
  const int kb0 = min(split * g.kper, kb_total);
  // the host never plans more than SKN_KMAX of K per workgroup; the clamp keeps
  // the LDS slice in bounds regardless
  const int kb1 = min(min(kb0 + g.kper, kb_total), kb0 + SKN_KMAX / 32);
  const int64_t kbeg = (int64_t)kb0 * 32;
  const int nkc = (kb1 - kb0) * 4;  // 8-k chunks of this workgroup

  // Stage B^T: block (kc, ng) = rows kbeg + 8kc .. +7, columns 8ng .. 8ng+7.
  for (int blk = tid; blk < nkc * (NCOL / 8); blk += 256) {
    const int ng = blk % (NCOL / 8), kc = blk / (NCOL / 8);
    const int64_t n = (int64_t)ng * 8;
    u32x4 r[8], c[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t k = kbeg + kc * 8 + i;
      r[i] = (k < K) ? load16_guard(g.B + k * ldb + n, N - n) : u32x4{0u, 0u, 0u, 0u};
    }
    transpose8x8(r, c);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int nn = ng * 8 + j;
      sBt[nn * KCH + (kc ^ (nn & 15))] = c[j];
    }
  }
  __syncthreads();

  f32x4 acc[RB][NT];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[rb][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int64_t row0 = (int64_t)rbk * (64 * RB) + wave * (16 * RB) + (lane & 15);
  const int kg = lane >> 4;
  for (int kb = kb0; kb < kb1; kb += U) {
    u32x4 fa[U][RB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t k = (int64_t)(kb + u) * 32 + kg * 8;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int64_t row = row0 + rb * 16;
        fa[u][rb] = (kb + u < kb1 && row < M) ? load16_guard(g.A + row * lda + k, K - k) : u32x4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (kb + u >= kb1) break;
      const int kc = (kb + u - kb0) * 4 + kg;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int nn = nt * 16 + (lane & 15);
        const u32x4 fb = sBt[nn * KCH + (kc ^ (nn & 15))];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) acc[rb][nt] = mfma16(fa[u][rb], fb, acc[rb][nt]);
      }
    }
  }

  // Output: lane holds column nt*16 + l%16 of rows base + rb*16 + 4*(l/16) + r.
  auto store_out = [&](const f32x4 (&v)[RB][NT]) {
    const int64_t rbase = (int64_t)rbk * (64 * RB) + wave * (16 * RB) + (lane >> 4) * 4;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int64_t col = nt * 16 + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = rbase + rb * 16 + r;
          if (row < M && col < N) store_c<OBF>(g.C, row * g.ldc + col, v[rb][nt][r]);
        }
      }
  };

  if (g.pk == 1) {
    store_out(acc);
    return;
  }
  const size_t blk_floats = (size_t)4 * RB * NT * 64 * 4;
  float* wblk = g.ws + (size_t)rbk * g.pk * blk_floats;
  {
    float* mine = wblk + (size_t)split * blk_floats;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        *reinterpret_cast<f32x4*>(mine + (((size_t)(wave * RB + rb) * NT + nt) * 64 + lane) * 4) = acc[rb][nt];
  }
  if (!arrive_last(g.counters + rbk, g.pk, &s_flag)) return;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const size_t off = (((size_t)(wave * RB + rb) * NT + nt) * 64 + lane) * 4;
      f32x4 s = *reinterpret_cast<const f32x4*>(wblk + off);
      for (int p = 1; p < g.pk; ++p) s += *reinterpret_cast<const f32x4*>(wblk + p * blk_floats + off);
      acc[rb][nt] = s;
    }
  store_out(acc);
}

}  // namespace ac

// ------------------------------------------------------------- registry
// VariantKey (family, config, output type) -> kernel; the launch boundary
// between the host planner and the device.
#include "planner.h"
#include "registry.h"

namespace ac {

namespace {

typedef hipError_t (*LaunchFn)(const Plan&, const GemmArgs&, hipStream_t, bool);
typedef int (*OccFn)();

template <int BM, int BN, int MS>
hipError_t launch_tile(const Plan& p, const GemmArgs& g, hipStream_t st, bool obf) {
  const dim3 grid(p.grid_x, p.grid_y), block(256);
  if (obf)
    hipLaunchKernelGGL((k_tile<BM, BN, MS, true>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_tile<BM, BN, MS, false>), grid, block, 0, st, g);
  return hipGetLastError();
}
template <int BM, int BN, int MS>
hipError_t launch_streamk(const Plan& p, const GemmArgs& g, hipStream_t st, bool obf) {
  const dim3 grid(p.grid_x, 1), block(256);
  if (obf)
    hipLaunchKernelGGL((k_streamk<BM, BN, MS, true>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_streamk<BM, BN, MS, false>), grid, block, 0, st, g);
  return hipGetLastError();
}
template <int MT, int WKW>
hipError_t launch_skinny_m(const Plan& p, const GemmArgs& g, hipStream_t st, bool obf) {
  const dim3 grid(p.grid_x, p.grid_y), block(256);
  if (obf)
    hipLaunchKernelGGL((k_skinny_m<MT, WKW, true>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_skinny_m<MT, WKW, false>), grid, block, 0, st, g);
  return hipGetLastError();
}
template <int NT, int RB>
hipError_t launch_skinny_n(const Plan& p, const GemmArgs& g, hipStream_t st, bool obf) {
  const dim3 grid(p.grid_x, p.grid_y), block(256);
  if (obf)
    hipLaunchKernelGGL((k_skinny_n<NT, RB, true>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_skinny_n<NT, RB, false>), grid, block, 0, st, g);
  return hipGetLastError();
}

template <typename F>
int occ_of(F kernel_f32, F kernel_bf16) {
  int a = 0, b = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&a, reinterpret_cast<const void*>(kernel_f32), 256, 0) != hipSuccess)
    a = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, reinterpret_cast<const void*>(kernel_bf16), 256, 0) != hipSuccess)
    b = 0;
  return a < b ? a : b;
}
template <int BM, int BN, int MS>
int occ_tile() {
  return occ_of(k_tile<BM, BN, MS, false>, k_tile<BM, BN, MS, true>);
}
template <int BM, int BN, int MS>
int occ_streamk() {
  return occ_of(k_streamk<BM, BN, MS, false>, k_streamk<BM, BN, MS, true>);
}
template <int MT, int WKW>
int occ_skinny_m() {
  return occ_of(k_skinny_m<MT, WKW, false>, k_skinny_m<MT, WKW, true>);
}
template <int NT, int RB>
int occ_skinny_n() {
  return occ_of(k_skinny_n<NT, RB, false>, k_skinny_n<NT, RB, true>);
}

#define TILES(X) X(256, 256, 32), X(256, 128, 32), X(128, 256, 32), X(128, 128, 32), \
                 X(128, 64, 32), X(64, 128, 32), X(64, 64, 32), X(32, 32, 16)
#define L_TILE(a, b, c) &launch_tile<a, b, c>
#define L_SK(a, b, c) &launch_streamk<a, b, c>
#define O_TILE(a, b, c) &occ_tile<a, b, c>
#define O_SK(a, b, c) &occ_streamk<a, b, c>
const LaunchFn kTileFns[] = {TILES(L_TILE)};
const LaunchFn kStreamKFns[] = {TILES(L_SK)};
const OccFn kTileOcc[] = {TILES(O_TILE)};
const OccFn kStreamKOcc[] = {TILES(O_SK)};
const LaunchFn kSkinnyMFns[] = {&launch_skinny_m<1, 1>, &launch_skinny_m<1, 4>, &launch_skinny_m<2, 1>,
                                &launch_skinny_m<2, 4>, &launch_skinny_m<4, 1>, &launch_skinny_m<4, 4>};
const OccFn kSkinnyMOcc[] = {&occ_skinny_m<1, 1>, &occ_skinny_m<1, 4>, &occ_skinny_m<2, 1>,
                             &occ_skinny_m<2, 4>, &occ_skinny_m<4, 1>, &occ_skinny_m<4, 4>};
const LaunchFn kSkinnyNFns[] = {&launch_skinny_n<1, 2>, &launch_skinny_n<2, 2>, &launch_skinny_n<4, 2>};
const OccFn kSkinnyNOcc[] = {&occ_skinny_n<1, 2>, &occ_skinny_n<2, 2>, &occ_skinny_n<4, 2>};
static_assert(sizeof(kTileFns) / sizeof(kTileFns[0]) == N_TILE_CFG, "tile table");
static_assert(sizeof(kSkinnyMFns) / sizeof(kSkinnyMFns[0]) == N_SKINNY_M_CFG, "skinny-M table");
static_assert(sizeof(kSkinnyNFns) / sizeof(kSkinnyNFns[0]) == N_SKINNY_N_CFG, "skinny-N table");

// The tables above must list the configurations in the order of variants.h.
constexpr bool tile_order_ok() {
  const int e[][3] = {{256, 256, 32}, {256, 128, 32}, {128, 256, 32}, {128, 128, 32},
                      {128, 64, 32},  {64, 128, 32},  {64, 64, 32},   {32, 32, 16}};
  for (int i = 0; i < N_TILE_CFG; ++i)
    if (kTileCfg[i].bm != e[i][0] || kTileCfg[i].bn != e[i][1] || kTileCfg[i].ms != e[i][2]) return false;
  return true;
}
static_assert(tile_order_ok(), "tile configuration order");
static_assert(kSkinnyMCfg[0].mt == 1 && kSkinnyMCfg[1].wkw == 4 && kSkinnyMCfg[4].mt == 4, "skinny-M order");
static_assert(kSkinnyNCfg[0].nt == 1 && kSkinnyNCfg[2].nt == 4 && kSkinnyNCfg[0].rb == 2, "skinny-N order");
static_assert(SKINNY_N_KMAX == SKN_KMAX, "skinny-N LDS slice");

}  // namespace

hipError_t launch_plan(const Plan& p, const GemmArgs& g, hipStream_t st) {
  const bool obf = p.s.dtype == AC_BF16_BF16OUT;
  switch (p.family) {
    case FAM_TILE:
      return kTileFns[p.cfg](p, g, st, obf);
    case FAM_STREAMK:
      return kStreamKFns[p.cfg](p, g, st, obf);
    case FAM_SKINNY_M:
      return kSkinnyMFns[p.cfg](p, g, st, obf);
    case FAM_SKINNY_N:
      return kSkinnyNFns[p.cfg](p, g, st, obf);
  }
  return hipErrorInvalidValue;
}

void query_occupancy() {
  for (int i = 0; i < N_TILE_CFG; ++i) {
    set_runtime_occupancy(FAM_TILE, i, kTileOcc[i]());
    set_runtime_occupancy(FAM_STREAMK, i, kStreamKOcc[i]());
  }
  for (int i = 0; i < N_SKINNY_M_CFG; ++i) set_runtime_occupancy(FAM_SKINNY_M, i, kSkinnyMOcc[i]());
  for (int i = 0; i < N_SKINNY_N_CFG; ++i) set_runtime_occupancy(FAM_SKINNY_N, i, kSkinnyNOcc[i]());
}

}  // namespace ac
