// gfx950 macro-tile kernels whose operand tiles travel from global memory
// straight into LDS (buffer_load ... lds: no staging registers, no register
// transposes) through S LDS stages, so that S - 1 k-blocks of loads are in
// flight while one is multiplied out (the Multi-Buffer module of Table 2;
// the schedule of Eq. 13 with a deeper pipeline).
//
//   A tile  BM x 64 k, row-major as in memory, 16-byte chunks XOR-swizzled
//           per row; MFMA fragments read with ds_read_b128.
//   B tile  64 k x BN, row-major as in memory (chunks swizzled per k-row);
//           MFMA fragments read with the LDS transpose read
//           ds_read_b64_tr_b16, which hands each lane four consecutive k of
//           one column: the k-contiguous operand the MFMA needs, without the
//           v_perm transposes of the register-staged kernel.
//   C       4 waves in a 2 x 2 grid, each a (BM/2) x (BN/2) quadrant of
//           32 x 32 x 16 MFMAs (tiles of at most 64 rows: 4 waves side by
//           side along N); fp32 accumulation in the accumulation registers;
//           bf16 output converted through a per-wave LDS slab and written as
//           whole 16-byte row segments.
//
// The swizzle of a stage is applied on the global side: a wave-wide LDS load
// writes 1024 contiguous bytes (lane l to bytes 16l .. 16l+15), so each lane
// fetches the global chunk that belongs at its slot.
//
// k_dl needs row-major operands with 16-byte aligned rows (A and B base
// addresses 16-byte aligned, lda and ldb multiples of 8 below 2^22) and K, N
// multiples of 8. A plan for other shapes either copies the operand
// zero-padded first (k_pad16 below, the Padding module) or runs k_dlu, the
// register-load form of the same tiling (16-byte loads at any 2-byte
// alignment, two LDS stages); an operand found misaligned at run time takes
// k_dlu, or the register-staged tile kernel of the same tiling where the
// configuration has no k_dlu. Chunks outside the matrices (rows past M,
// columns past N, k past K) are read as zeros through out-of-range buffer
// offsets, so edge tiles take the same path.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "kernel_args.h"
#include "registry.h"

#ifndef AC_INPUT_F16
#define AC_INPUT_F16 0
#endif

namespace ac {
#if AC_INPUT_F16
namespace f16 {
#endif

#include "device_common.h"

namespace {

// the transpose read moves 16-bit patterns; its bf16 form serves fp16 too
typedef __bf16 tr16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) tr16x4 lds_tr16x4;

enum DlOut : int { DL_F32 = 0, DL_BF16 = 1, DL_PARTIAL = 2 };

template <int BM, int BN, int BK_, int S_>
struct Dl {
  static constexpr int BN_ = BN, BK = BK_, S = S_, NT = 256;
  // waves: 2 x 2 quadrants, or (tiles of at most 64 rows: the decode-style
  // shapes) 1 x 4 along N
  static constexpr int WM = BM >= 128 ? 2 : 1, WN = 4 / WM;
  static constexpr int WTM = BM / WM, WTN = BN / WN;  // a wave's part of the tile
  static constexpr int TM = WTM / 32, TN = WTN / 32;
  static constexpr int A_BYTES = BM * BK * 2, B_BYTES = BK * BN * 2;
  static constexpr int A_LPR = BK / 8;        // 16-byte chunks of an A row
  static constexpr int A_RPI = 64 / A_LPR;    // A rows per wave-wide load
  static constexpr int B_LPR = BN / 8;        // 16-byte chunks of a B row
  static constexpr int B_RPI = 64 / B_LPR;    // B rows per wave-wide load
  static constexpr int NIA = A_BYTES / 4096;  // wave-wide loads per wave and A stage
  static constexpr int NIB = B_BYTES / 4096;
  static constexpr int LOADS = NIA + NIB;
  static constexpr int CT_LD = WTN + 4;       // padded row of the bf16 output slab
  // workgroups per CU the configuration is built for: two when two fit the
  // LDS and the register file (two waves per SIMD, at most 256 registers
  // each): one workgroup's epilogue stores then overlap the other's loads
  // and MFMAs
  static constexpr int WPE = (S * (BM + BN) * BK * 2 <= 80 * 1024 && BM * BN <= 256 * 128) ? 2 : 1;
  static_assert(BM % 32 == 0 && BM >= 32 && BN >= 128 && BN <= 512 && (BK == 32 || BK == 64) && WTN % 32 == 0,
                "tile");
  static_assert(3 * LOADS <= 63, "vmcnt range");
  // the bf16 epilogue's per-wave slab of 32 output rows goes into one stage
  // buffer per wave: A0, A1, B0, B1 if both kinds are large enough, else
  // the first four of the kind that is, else two slabs in each of B0, B1
  static constexpr int SLAB = 32 * CT_LD * 2;
  static constexpr int SLAB_KIND = (SLAB <= A_BYTES && SLAB <= B_BYTES) ? 0
                                   : (SLAB <= B_BYTES && S >= 4)        ? 1
                                   : (2 * SLAB <= B_BYTES)              ? 3
                                                                        : 2;
  static_assert(SLAB_KIND != 2 || (SLAB <= A_BYTES && S >= 4), "output slab fits a stage buffer");
};

// B stage: chunk c of k-row r sits at slot c ^ f(r & 3), f = 0, 6, 12, 10.
// One transpose read covers 4 consecutive k-rows and 2 (16 lanes) or 4 (32
// lanes) consecutive chunks; f keeps those on distinct banks for both 32
// and 64 banks.
__device__ __forceinline__ int swz_b(int r) { return (0xAC60 >> (4 * (r & 3))) & 15; }

// Workgroup barrier of the pipeline: this wave waits until at most `ahead`
// (0 .. 3) later stages of its own loads are in flight and its LDS reads
// are done, then all waves meet. After it every wave's loads of the stage
// about to be read have landed and no wave still reads the stage about to be
// reloaded. (__syncthreads would add a workgroup fence, which waits for ALL
// loads into LDS, the prefetched stages included.) The empty asm with a
// memory clobber keeps the compiler from moving LDS accesses across it.
template <int LOADS>
__device__ __forceinline__ void stage_barrier(int ahead) {
  if (ahead <= 0)
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  else if (ahead == 1)
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(LOADS));
  else if (ahead == 2)
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * LOADS));
  else
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(3 * LOADS));
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Per-tile addressing of a workgroup's loads: the byte offset of every
// 16-byte chunk this lane loads (OOB_OFF for rows past M and columns past
// N), and the k of that chunk within the block for the K tail.
template <class G>
struct DlTile {
  const char* a;  // A + m0 * lda
  const char* b;  // B + n0
  int64_t ldb2;
  int64_t K, kB;  // k of the loop (A's columns), rows of B
  int32_t a_off[G::NIA], b_off[G::NIB];
  int32_t a_k[G::NIA], b_k[G::NIB];

  __device__ __forceinline__ void init(const GemmArgs& g, int64_t m0, int64_t n0) {
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    a = reinterpret_cast<const char*>(g.A + m0 * g.lda);
    b = reinterpret_cast<const char*>(g.B + n0);
    ldb2 = g.ldb * 2;
    K = g.K;
    kB = g.kB;
    const int64_t rows = g.M - m0, cols = g.nB - n0;
#pragma unroll
    for (int q = 0; q < G::NIA; ++q) {
      const int u = w * G::NIA + q;            // 1024-byte block of the stage: A_RPI rows
      const int row = u * G::A_RPI + lane / G::A_LPR;
      const int c = (lane % G::A_LPR) ^ swz_a<G::BK>(row);  // the chunk this slot holds
      a_off[q] = row < rows ? (int32_t)(row * g.lda * 2) + c * 16 : OOB_OFF;
      a_k[q] = c * 8;
    }
#pragma unroll
    for (int q = 0; q < G::NIB; ++q) {
      const int u = w * G::NIB + q;
      const int kr = u * G::B_RPI + lane / G::B_LPR;
      const int c = (lane % G::B_LPR) ^ swz_b(kr);
      b_off[q] = c * 8 < cols ? (int32_t)(kr * g.ldb * 2) + c * 16 : OOB_OFF;
      b_k[q] = kr;
    }
  }
};

// This wave's share of the loads of one k-block (starting at k0) into one
// stage: NIA loads of A, then NIB loads of B, issued one at a time so that
// they can be spread between MFMAs. A block past K (the pipeline's tail)
// loads nothing: every offset is out of range, the stage gets zeros that no
// step reads.
template <class G>
struct StageLoads {
  __amdgpu_buffer_rsrc_t ra, rb;
  char* sA;
  char* sB;
  int krem, kremB;
  bool full, fullB;
  __device__ __forceinline__ void init(char* a_stage, char* b_stage, const DlTile<G>& t, int64_t k0) {
    const int64_t kleft = t.K - k0, kleftB = t.kB - k0;
    krem = kleft < G::BK ? (int)(kleft > 0 ? kleft : 0) : G::BK;  // k of A in this block (uniform)
    kremB = kleftB < G::BK ? (int)(kleftB > 0 ? kleftB : 0) : G::BK;  // rows of B in this block
    full = krem == G::BK;  // only a K tail needs the per-chunk test
    fullB = kremB == G::BK;
    ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(t.a) + k0 * 2, (short)0, (int)0x7FFFFFF0,
                                           (int)RSRC_WORD3);
    rb = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(t.b) + k0 * t.ldb2, (short)0, (int)0x7FFFFFF0,
                                           (int)RSRC_WORD3);
    sA = a_stage;
    sB = b_stage;
  }
  // load q of this wave (0 .. NIA + NIB - 1; a compile-time index)
  __device__ __forceinline__ void issue(const DlTile<G>& t, int q) const {
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (q < G::NIA) {
      const int32_t off = full || t.a_k[q] < krem ? t.a_off[q] : OOB_OFF;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(sA + (w * G::NIA + q) * 1024), 16, off, 0, 0, 0);
    } else {
      const int qb = q - G::NIA;
      const int32_t off = fullB || t.b_k[qb] < kremB ? t.b_off[qb] : OOB_OFF;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void*)(sB + (w * G::NIB + qb) * 1024), 16, off, 0, 0, 0);
    }
  }
};

template <class G>
__device__ __forceinline__ void issue_stage(char* sA, char* sB, const DlTile<G>& t, int64_t k0) {
  StageLoads<G> L;
  L.init(sA, sB, t, k0);
#pragma unroll
  for (int q = 0; q < G::LOADS; ++q) L.issue(t, q);
}

// ---- loads through registers (any alignment, K >= 8 and N >= 8)
// The same chunks into the same LDS slots as the direct loads, fetched with
// 16-byte loads at any 2-byte address: a chunk that crosses the end of a
// row is loaded as the 16 bytes ending at the row end and shifted down in
// registers, with zeros past K (A columns, B rows) and past N (B columns).
// Rows past M re-read row M - 1 (their outputs are never stored).
template <class G>
struct DlTileU {
  const uint16_t* a;  // A + m0 * lda
  const uint16_t* B;
  int64_t ldb, K, N;
  uint32_t a_row[G::NIA];  // bytes: clamped row * lda * 2
  int32_t a_c[G::NIA];     // k of the chunk within the block
  int32_t b_kr[G::NIB];    // k-row of the chunk within the block
  uint32_t b_col[G::NIB];  // bytes: first column loaded (<= N - 8)
  int32_t b_cs[G::NIB];    // elements dropped at the N edge (0 .. 8)

  __device__ __forceinline__ void init(const GemmArgs& g, int64_t m0, int64_t n0) {
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    a = g.A + m0 * g.lda;
    B = g.B;
    ldb = g.ldb;
    K = g.K;
    N = g.N;
#pragma unroll
    for (int q = 0; q < G::NIA; ++q) {
      const int u = w * G::NIA + q;
      const int row = u * G::A_RPI + lane / G::A_LPR;
      const int c = (lane % G::A_LPR) ^ swz_a<G::BK>(row);
      a_row[q] = (uint32_t)((min(m0 + row, g.M - 1) - m0) * g.lda * 2);
      a_c[q] = c * 8;
    }
#pragma unroll
    for (int q = 0; q < G::NIB; ++q) {
      const int u = w * G::NIB + q;
      const int kr = u * G::B_RPI + lane / G::B_LPR;
      const int c = (lane % G::B_LPR) ^ swz_b(kr);
      const int64_t gn = n0 + c * 8, st = min(gn, g.N - 8);
      b_kr[q] = kr;
      b_col[q] = (uint32_t)(st * 2);
      b_cs[q] = (int32_t)min(gn - st, (int64_t)8);
    }
  }
};

template <class G>
struct RegLoads {
  u32x4 va[G::NIA], vb[G::NIB];
  uint32_t sha, shb;  // per chunk 4 bits: elements to drop (8 = all)
  const uint16_t* a0;  // A tile base at this block's k (elements: the chunk's start added per lane)
  const uint16_t* b0;  // B + min(k0, K - 1) * ldb
  int64_t k0, kb0;
  char* sA;
  char* sB;
  __device__ __forceinline__ void init(char* a_stage, char* b_stage, const DlTileU<G>& t, int64_t k) {
    k0 = k;
    kb0 = min(k, t.K - 1);
    b0 = t.B + kb0 * t.ldb;
    sA = a_stage;
    sB = b_stage;
    sha = shb = 0;
  }
  // global load q into registers (0 .. NIA + NIB - 1, a compile-time index)
  __device__ __forceinline__ void issue(const DlTileU<G>& t, int q) {
    if (q < G::NIA) {
      const int64_t e = k0 + t.a_c[q], st = min(e, t.K - 8);
      const uint32_t s = (uint32_t)min(e - st, (int64_t)8);
      va[q] = load16(reinterpret_cast<const uint16_t*>(reinterpret_cast<const char*>(t.a) + t.a_row[q] + st * 2));
      sha |= s << (4 * q);
    } else {
      const int qb = q - G::NIA;
      const int64_t r = k0 + t.b_kr[qb];
      const int64_t rr = min(r, t.K - 1) - kb0;  // >= 0
      vb[qb] = load16(reinterpret_cast<const uint16_t*>(reinterpret_cast<const char*>(b0) +
                                                         (uint32_t)(rr * t.ldb * 2) + t.b_col[qb]));
      const uint32_t s = r >= t.K ? 8u : (uint32_t)t.b_cs[qb];
      shb |= s << (4 * qb);
    }
  }
  // the shifted chunks into their LDS slots (after the loads landed)
  __device__ __forceinline__ void finish() {
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int q = 0; q < G::NIA; ++q)
      *reinterpret_cast<u32x4*>(sA + (w * G::NIA + q) * 1024 + lane * 16) = shift_down(va[q], (sha >> (4 * q)) & 15);
#pragma unroll
    for (int q = 0; q < G::NIB; ++q)
      *reinterpret_cast<u32x4*>(sB + (w * G::NIB + q) * 1024 + lane * 16) = shift_down(vb[q], (shb >> (4 * q)) & 15);
  }
};

// Fragments of one k-step (16 k) of a stage: TM A fragments (ds_read_b128
// of a swizzled row chunk) and TN B fragments (two transpose reads each).
template <class G>
struct Frags {
  u32x4 a[G::TM], b[G::TN];
};

template <class G>
__device__ __forceinline__ void read_frags(const char* sA, const char* sB, int ks, int wr, int wc, Frags<G>& f) {
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31, hi = lane >> 5, i16 = lane & 15, g = lane >> 4;
#pragma unroll
  for (int i = 0; i < G::TM; ++i) {
    const int row = wr * G::WTM + 32 * i + l32;
    const int ch = 2 * ks + hi;  // 8 consecutive k of the lane's k-group
    f.a[i] = *reinterpret_cast<const u32x4*>(sA + row * (G::BK * 2) + ((ch ^ swz_a<G::BK>(row)) << 4));
  }
  // the transpose read of a 16-lane group covers 4 k-rows x 16 columns: lane
  // i16 addresses k-row i16 >> 2 and columns 4 * (i16 & 3) .. +3 and receives
  // column i16 of the 4 rows; groups 0 / 1 take columns 0-15 / 16-31 of the
  // fragment at the lane's k-group 0, groups 2 / 3 the same at k-group 1
  const int kr0 = 8 * (g >> 1) + (i16 >> 2);
  const int sw = swz_b(kr0);  // every k-row the lane reads is kr0 mod 4
#pragma unroll
  for (int j = 0; j < G::TN; ++j) {
    const int col = wc * G::WTN + 32 * j + 16 * (g & 1) + (i16 & 3) * 4;
    const int cb = ((col >> 3) ^ sw) * 16 + (col & 7) * 2;
    uint32_t v[4];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int kr = 16 * ks + 4 * h + kr0;
      const tr16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_tr16x4*)(sB + kr * (G::BN_ * 2) + cb));
      const uint64_t bits = __builtin_bit_cast(uint64_t, r);
      v[2 * h] = (uint32_t)bits;
      v[2 * h + 1] = (uint32_t)(bits >> 32);
    }
    f.b[j] = u32x4{v[0], v[1], v[2], v[3]};
  }
}

// Multiplies out one stage: BK / 16 k-steps, TM x TN MFMAs each, while the
// next stage's loads go out. The reads of step ks + 1 are issued before the
// MFMAs of step ks (two fragment sets), so their latency runs under those
// MFMAs; the next stage's global loads are spread one per MFMA over the
// steps instead of leaving in one burst (a burst fills the load queue, and
// a wave stalled on a full queue issues no MFMAs). The scheduling barriers
// keep the compiler to this order.
template <class G, class Loads, class Tile>
__device__ __forceinline__ void compute_stage(const char* sA, const char* sB, f32x16 (&acc)[G::TM][G::TN],
                                              int wr, int wc, Loads& nxt, const Tile& t) {
  constexpr int KS = G::BK / 16, NMF = G::TM * G::TN;
  // next-stage loads per k-step: with two stages the loads must land
  // within this stage, so they all go out as early as possible (one per
  // MFMA from the first step on); with more stages they are spread evenly
  constexpr int LPS = G::S == 2 ? NMF : (G::LOADS + KS - 1) / KS;
  static_assert(G::S > 2 || G::LOADS <= KS * NMF, "one load per MFMA at most");
  Frags<G> f[2];
  read_frags<G>(sA, sB, 0, wr, wc, f[0]);
  __builtin_amdgcn_sched_barrier(0);  // step 0's reads first: its MFMAs wait for those only
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    Frags<G>& cur = f[ks & 1];
    if (ks + 1 < KS) read_frags<G>(sA, sB, ks + 1, wr, wc, f[(ks + 1) & 1]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < G::TM; ++i)
#pragma unroll
      for (int j = 0; j < G::TN; ++j) acc[i][j] = mfma32(cur.b[j], cur.a[i], acc[i][j]);  // C^T: a lane holds a row of C
#pragma unroll
    for (int q = ks * LPS; q < (ks + 1) * LPS && q < G::LOADS; ++q) nxt.issue(t, q);
#pragma unroll
    for (int m = 0; m < NMF; ++m) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
      if (m < LPS && ks * LPS + m < G::LOADS) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // one load
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (std::is_same<Loads, RegLoads<G>>::value) nxt.finish();  // registers -> the next stage
}

// One output tile (tile coordinates tm, tn) over K partition `split` of the
// plan's kper-block partitions.
template <int BM, int BN, int BK, int S, int OUT, bool RG>
__device__ __forceinline__ void dl_tile(const GemmArgs& g, int tm, int tn, int split) {
  typedef Dl<BM, BN, BK, S> G;
  typedef typename std::conditional<RG, DlTileU<G>, DlTile<G>>::type Tile;
  typedef typename std::conditional<RG, RegLoads<G>, StageLoads<G>>::type Loads;
  __shared__ __attribute__((aligned(1024))) char lA0[G::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char lA1[G::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char lA2[G::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char lA3[G::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char lA4[G::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char lB0[G::B_BYTES];
  __shared__ __attribute__((aligned(1024))) char lB1[G::B_BYTES];
  __shared__ __attribute__((aligned(1024))) char lB2[G::B_BYTES];
  __shared__ __attribute__((aligned(1024))) char lB3[G::B_BYTES];
  __shared__ __attribute__((aligned(1024))) char lB4[G::B_BYTES];
  static_assert(S >= 2 && S <= 5, "stages");

  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  // the K partition: kper blocks of the plan's 64-deep granule, a whole
  // number of this kernel's k-blocks
  const int64_t kbeg = min((int64_t)split * g.kper * 64, g.K);
  const int64_t kend = min(kbeg + (int64_t)g.kper * 64, g.K);
  const int nk = (int)((kend - kbeg + G::BK - 1) / G::BK);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wr = wave / G::WN, wc = wave % G::WN;

  Tile t;
  t.init(g, m0, n0);

  f32x16 acc[G::TM][G::TN];
#pragma unroll
  for (int i = 0; i < G::TM; ++i)
#pragma unroll
    for (int j = 0; j < G::TN; ++j) acc[i][j] = f32x16{};

  // Stage I holds k-blocks I, I + S, I + 2S, ... of the partition. The
  // stage buffers are distinct variables so that the compiler's wait
  // before a read of one stage does not include the loads into the others.
  auto stA = [&](auto ic) -> char* {
    constexpr int I = decltype(ic)::value;
    return I == 0 ? lA0 : I == 1 ? lA1 : I == 2 ? lA2 : I == 3 ? lA3 : lA4;
  };
  auto stB = [&](auto ic) -> char* {
    constexpr int I = decltype(ic)::value;
    return I == 0 ? lB0 : I == 1 ? lB1 : I == 2 ? lB2 : I == 3 ? lB3 : lB4;
  };
  // Every step issues one stage of loads (past the partition's last block:
  // out-of-range loads), so at step kb exactly S - 2 stages of this wave's
  // loads were issued after those of block kb.
  const int64_t kstop = kbeg + (int64_t)nk * G::BK;  // the partition's end, rounded up to a block
  auto kpos = [&](int b) { const int64_t k = kbeg + (int64_t)b * G::BK; return k < kstop ? k : t.K; };
  auto prologue = [&](char* a_st, char* b_st, int64_t k) {
    Loads L;
    L.init(a_st, b_st, t, k);
#pragma unroll
    for (int q = 0; q < G::LOADS; ++q) L.issue(t, q);
    if constexpr (RG) L.finish();
  };
  if (nk > 0) {
    prologue(lA0, lB0, kpos(0));
    if constexpr (S > 2) prologue(lA1, lB1, kpos(1));
    if constexpr (S > 3) prologue(lA2, lB2, kpos(2));
    if constexpr (S > 4) prologue(lA3, lB3, kpos(3));
  }

  auto step = [&](auto ic, int kb) {
    constexpr int I = decltype(ic)::value;
    constexpr int NX = (I + S - 1) % S;  // stage that receives block kb + S - 1
    stage_barrier<G::LOADS>(RG ? 0 : S - 2);
    Loads nxt;
    nxt.init(stA(std::integral_constant<int, NX>{}), stB(std::integral_constant<int, NX>{}), t, kpos(kb + S - 1));
    compute_stage<G>(stA(ic), stB(ic), acc, wr, wc, nxt, t);
  };
  // whole groups of S blocks, then the remaining 0 .. S-1 blocks
  int kb = 0;
  for (; kb + S <= nk; kb += S) {
    step(std::integral_constant<int, 0>{}, kb);
    step(std::integral_constant<int, 1>{}, kb + 1);
    if constexpr (S > 2) step(std::integral_constant<int, 2>{}, kb + 2);
    if constexpr (S > 3) step(std::integral_constant<int, 3>{}, kb + 3);
    if constexpr (S > 4) step(std::integral_constant<int, 4>{}, kb + 4);
  }
  if (kb < nk) step(std::integral_constant<int, 0>{}, kb);
  if (kb + 1 < nk) step(std::integral_constant<int, 1>{}, kb + 1);
  if constexpr (S > 3)
    if (kb + 2 < nk) step(std::integral_constant<int, 2>{}, kb + 2);
  if constexpr (S > 4)
    if (kb + 3 < nk) step(std::integral_constant<int, 3>{}, kb + 3);

  // ---- epilogue
  const int64_t rbase = m0 + wr * G::WTM, cbase = n0 + wc * G::WTN;
  if constexpr (OUT == DL_BF16) {
    stage_barrier<G::LOADS>(0);  // every wave's last reads of the stages are done
    // the wave's slab: 32 rows x WTN bf16 in one of the stage buffers
    char* slab;
    if constexpr (G::SLAB_KIND == 0)
      slab = wave == 0 ? lA0 : wave == 1 ? lA1 : wave == 2 ? lB0 : lB1;
    else if constexpr (G::SLAB_KIND == 1)
      slab = wave == 0 ? lB0 : wave == 1 ? lB1 : wave == 2 ? lB2 : lB3;
    else if constexpr (G::SLAB_KIND == 3)
      slab = (wave < 2 ? lB0 : lB1) + (wave & 1) * G::SLAB;
    else
      slab = wave == 0 ? lA0 : wave == 1 ? lA1 : wave == 2 ? lA2 : lA3;
    uint16_t* ct = reinterpret_cast<uint16_t*>(slab);
    uint16_t* C = static_cast<uint16_t*>(g.C);
    constexpr int GPR = G::WTN / 8;  // 16-byte groups per slab row
#pragma unroll
    for (int i = 0; i < G::TM; ++i) {
      const int64_t row = rbase + 32 * i + (lane & 31);
#pragma unroll
      for (int j = 0; j < G::TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = 32 * j + (q << 3) + ((lane >> 5) << 2);  // acc elements 4q .. 4q+3: four columns
          float w[4] = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
          if (g.epi && row < g.M && cbase + c < g.N) epi_apply<true, 4>(g, w, row, cbase + c, g.N - cbase - c);
          const uint32_t lo = (uint32_t)to16(w[0]) | ((uint32_t)to16(w[1]) << 16);
          const uint32_t hi = (uint32_t)to16(w[2]) | ((uint32_t)to16(w[3]) << 16);
          *reinterpret_cast<uint64_t*>(ct + (lane & 31) * G::CT_LD + c) = (uint64_t)lo | ((uint64_t)hi << 32);
        }
      // the slab back as 16-byte row segments (the same wave: LDS is in order)
#pragma unroll
      for (int v = 0; v < 32 * GPR / 64; ++v) {
        const int u = lane + 64 * v, r = u / GPR, grp = u % GPR;
        const uint16_t* src = ct + r * G::CT_LD + grp * 8;
        const uint64_t a = *reinterpret_cast<const uint64_t*>(src);
        const uint64_t b = *reinterpret_cast<const uint64_t*>(src + 4);
        const int64_t gr = rbase + 32 * i + r, gc = cbase + grp * 8;
        if (gr < g.M && gc + 8 <= g.N) {
          const uint64_t vv[2] = {a, b};
          __builtin_memcpy(C + gr * g.ldc + gc, vv, 16);
        } else if (gr < g.M && gc < g.N) {  // the last, partial group of a row
          const uint16_t* e = src;
          for (int j = 0; j < (int)(g.N - gc); ++j) C[gr * g.ldc + gc + j] = e[j];
        }
      }
      __builtin_amdgcn_sched_barrier(0);  // slab by slab: bounded live registers
    }
  } else {
    float* dst = OUT == DL_PARTIAL ? g.ws + (size_t)split * (size_t)g.M * (size_t)g.ldw : static_cast<float*>(g.C);
    const int64_t ld = OUT == DL_PARTIAL ? g.ldw : g.ldc;
#pragma unroll
    for (int i = 0; i < G::TM; ++i) {
      const int64_t row = rbase + 32 * i + (lane & 31);
      if (row >= g.M) continue;
#pragma unroll
      for (int j = 0; j < G::TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int64_t col = cbase + 32 * j + (q << 3) + ((lane >> 5) << 2);
          if (col >= g.N) continue;
          float w[4] = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
          if (OUT == DL_F32 && g.epi) epi_apply<false, 4>(g, w, row, col, g.N - col);
          if (col + 4 <= g.N) {
            const f32x4 vv = {w[0], w[1], w[2], w[3]};
            __builtin_memcpy(dst + row * ld + col, &vv, 16);
          } else {
            for (int e = 0; e < (int)(g.N - col); ++e) dst[row * ld + col + e] = w[e];
          }
        }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// a workgroup per output tile (blockIdx.x, in the plan's tile order) and K
// partition (blockIdx.y)
template <int BM, int BN, int BK, int S, int OUT, bool RG>
__device__ __forceinline__ void dl_kernel(const GemmArgs& g) {
  const int ntiles = g.tiles_m * g.tiles_n;
  int tile = blockIdx.x;
  if (g.swizzle) tile = xcd_remap(tile, ntiles);
  int tm, tn;
  tile_coords(tile, g.tiles_m, g.tiles_n, g.swizzle, tm, tn);
  dl_tile<BM, BN, BK, S, OUT, RG>(g, tm, tn, (int)blockIdx.y);
}

// the kernels: operand tiles loaded straight into LDS (k_dl), or through
// registers at any alignment (k_dlu)
template <int BM, int BN, int BK, int S, int OUT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(Dl<BM, BN, BK, S>::WPE, Dl<BM, BN, BK, S>::WPE)))
void k_dl(GemmArgs g) {
  dl_kernel<BM, BN, BK, S, OUT, false>(g);
}
template <int BM, int BN, int BK, int S, int OUT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(Dl<BM, BN, BK, S>::WPE, Dl<BM, BN, BK, S>::WPE)))
void k_dlu(GemmArgs g) {
  dl_kernel<BM, BN, BK, S, OUT, true>(g);
}

// Off-chip accumulation (the SingleCoreSplitK and HybridSplitK templates of
// Section 4.2; write volume of Eqs. 3 and 5): a workgroup owns a super-tile
// of two vertically adjacent tiles, 2BM x BN, whose fp32 accumulator does not
// fit the registers, and takes the plan's P_k k1-slices of K in order --
// all of them (gridDim.y = 1: SingleCoreSplitK) or its share of them
// (gridDim.y workgroups along K: HybridSplitK). For every slice it computes
// the upper tile, flushes its partial sums to the slice's fp32 partial buffer
// in the workspace, then the lower tile (whose B slice the upper one has just
// brought into the L2); the reduction kernel then adds the slices. Each tile
// of each slice is the direct-to-LDS tile kernel's own computation of that
// partition, so the result has the bits of the split-K plan with the same
// partitions.
template <int BM, int BN, int BK, int S>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(Dl<BM, BN, BK, S>::WPE, Dl<BM, BN, BK, S>::WPE)))
void k_dl_sc(GemmArgs g) {
  const int sup = blockIdx.x;
  const int stm = sup / g.tiles_n, tn = sup - stm * g.tiles_n;
  const int per = g.pk / (int)gridDim.y;  // slices of this workgroup
  for (int q = 0; q < per; ++q) {
    const int split = (int)blockIdx.y * per + q;
#pragma unroll 1
    for (int h = 0; h < 2; ++h) {
      const int tm = 2 * stm + h;
      if (tm >= g.tiles_m) break;
      // the previous tile's loads and stores are complete and no wave still
      // reads its LDS stages
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
      __syncthreads();
      dl_tile<BM, BN, BK, S, DL_PARTIAL, false>(g, tm, tn, split);
    }
  }
}

template <int BM, int BN, int BK, int S>
hipError_t launch_dl(const Plan& p, const GemmArgs& g, hipStream_t st, bool obf) {
  const dim3 grid(p.grid_x, p.grid_y), block(256);
  if (p.unal) {
    if constexpr (dl_has_unal(BM, BN, BK, S)) {
      if (p.pk > 1)
        hipLaunchKernelGGL((k_dlu<BM, BN, BK, S, DL_PARTIAL>), grid, block, 0, st, g);
      else if (obf)
        hipLaunchKernelGGL((k_dlu<BM, BN, BK, S, DL_BF16>), grid, block, 0, st, g);
      else
        hipLaunchKernelGGL((k_dlu<BM, BN, BK, S, DL_F32>), grid, block, 0, st, g);
    } else {
      return hipErrorInvalidValue;
    }
  } else if (p.pk > 1)
    hipLaunchKernelGGL((k_dl<BM, BN, BK, S, DL_PARTIAL>), grid, block, 0, st, g);
  else if (obf)
    hipLaunchKernelGGL((k_dl<BM, BN, BK, S, DL_BF16>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_dl<BM, BN, BK, S, DL_F32>), grid, block, 0, st, g);
  return hipGetLastError();
}

template <int BM, int BN, int BK, int S>
int occ_dl() {
  int o = 1 << 20;
  const void* ks[6] = {reinterpret_cast<const void*>(k_dl<BM, BN, BK, S, DL_F32>),
                       reinterpret_cast<const void*>(k_dl<BM, BN, BK, S, DL_BF16>),
                       reinterpret_cast<const void*>(k_dl<BM, BN, BK, S, DL_PARTIAL>), nullptr, nullptr, nullptr};
  if constexpr (dl_has_unal(BM, BN, BK, S)) {  // the register-load form: one occupancy for both
    ks[3] = reinterpret_cast<const void*>(k_dlu<BM, BN, BK, S, DL_F32>);
    ks[4] = reinterpret_cast<const void*>(k_dlu<BM, BN, BK, S, DL_BF16>);
    ks[5] = reinterpret_cast<const void*>(k_dlu<BM, BN, BK, S, DL_PARTIAL>);
  }
  for (const void* k : ks) {
    if (!k) continue;
    int a = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&a, k, 256, 0) != hipSuccess) a = 0;
    o = a < o ? a : o;
  }
  return o;
}

typedef hipError_t (*DlLaunchFn)(const Plan&, const GemmArgs&, hipStream_t, bool);
typedef int (*DlOccFn)();
#define DL_CFGS(X) X(256, 256, 64, 2), X(256, 128, 64, 3), X(128, 256, 64, 3), X(128, 128, 64, 3), X(256, 256, 32, 4), \
    X(256, 256, 32, 5), X(256, 128, 32, 4), X(128, 256, 32, 4), X(256, 128, 32, 2), X(128, 128, 64, 2),       \
    X(128, 128, 32, 2), X(32, 256, 64, 4), X(64, 256, 64, 4), X(32, 128, 64, 4), X(64, 512, 32, 2)
#define DL_L(a, b, c, d) &launch_dl<a, b, c, d>
#define DL_O(a, b, c, d) &occ_dl<a, b, c, d>
#define DL_C(a, b, c, d) {a, b, c, d}
const DlLaunchFn kDlFns[] = {DL_CFGS(DL_L)};
const DlOccFn kDlOcc[] = {DL_CFGS(DL_O)};
constexpr int kDlCheck[][4] = {DL_CFGS(DL_C)};
constexpr bool dl_match() {
  for (int i = 0; i < N_DL_CFG; ++i)
    if (kDlCheck[i][0] != kDlCfg[i].bm || kDlCheck[i][1] != kDlCfg[i].bn || kDlCheck[i][2] != kDlCfg[i].bk ||
        kDlCheck[i][3] != kDlCfg[i].stages)
      return false;
  return true;
}
static_assert(sizeof(kDlFns) / sizeof(kDlFns[0]) == N_DL_CFG && dl_match(), "kernels must follow kDlCfg");
#define DL_W(a, b, c, d) Dl<a, b, c, d>::WPE
constexpr int kDlWpe[] = {DL_CFGS(DL_W)};
constexpr bool dl_occ_match() {
  for (int i = 0; i < N_DL_CFG; ++i)
    if (kDlWpe[i] != kDlCfg[i].occ) return false;
  return true;
}
static_assert(dl_occ_match(), "the table's workgroups per CU must be those the kernels are built for");

// the off-chip accumulation kernels: super-tiles of the 256 x 256 tiles
// (DL configurations 0 and 4), whose 512 KiB fp32 accumulator exceeds the
// registers
template <int BM, int BN, int BK, int S>
hipError_t launch_dl_sc(const Plan& p, const GemmArgs& g, hipStream_t st) {
  hipLaunchKernelGGL((k_dl_sc<BM, BN, BK, S>), dim3(p.grid_x, p.grid_y), dim3(256), 0, st, g);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_dl_sc_main(const Plan& p, const GemmArgs& g, hipStream_t st) {
  const int cfg = p.cfg & 0xF, kc = 1 << (p.cfg >> 4);
  if (p.family != FAM_DLSC || (cfg != 0 && cfg != 4) || p.grid_y != kc || p.pk < 2 || p.pk % kc != 0 ||
      g.pk != p.pk || (int64_t)p.grid_x != (int64_t)((g.tiles_m + 1) / 2) * g.tiles_n || !ac::dl_operands_aligned(g))
    return hipErrorInvalidValue;
  return cfg == 0 ? launch_dl_sc<256, 256, 64, 2>(p, g, st) : launch_dl_sc<256, 256, 32, 4>(p, g, st);
}

hipError_t launch_dl_main(const Plan& p, const GemmArgs& g, hipStream_t st) {
  if (p.family != FAM_DL || p.cfg < 0 || p.cfg >= N_DL_CFG) return hipErrorInvalidValue;
  // the register-load form takes any alignment (K >= 8, N >= 8; two stages)
  if (p.unal ? (!kDlCfg[p.cfg].unal || g.K < 8 || g.N < 8) : !ac::dl_operands_aligned(g)) return hipErrorInvalidValue;
  return kDlFns[p.cfg](p, g, st, dtype_out16(p.s.dtype));
}

void query_occupancy_dl() {
  for (int i = 0; i < N_DL_CFG; ++i) set_runtime_occupancy(FAM_DL, i, kDlOcc[i]());
}

#if AC_INPUT_F16
}  // namespace f16
#else
bool dl_a_aligned(const void* A, int64_t lda, int64_t K) {
  return (reinterpret_cast<uintptr_t>(A) & 15) == 0 && (lda & 7) == 0 && (K & 7) == 0 && lda < DL_MAX_LD;
}
bool dl_b_aligned(const void* B, int64_t ldb, int64_t nB) {
  return (reinterpret_cast<uintptr_t>(B) & 15) == 0 && (ldb & 7) == 0 && (nB & 7) == 0 && ldb < DL_MAX_LD;
}
bool dl_operands_aligned(const GemmArgs& g) { return dl_a_aligned(g.A, g.lda, g.K) && dl_b_aligned(g.B, g.ldb, g.nB); }

// ---- padding prologue (the Padding module of Table 2)
// dst (rows x ld_dst, ld_dst = cols rounded up to 8, 16-byte aligned) =
// src (rows x cols, row pitch ld_src, any 2-byte alignment), zeros in the pad
// columns: every row of the copy is a whole number of aligned 16-byte
// chunks. A thread moves one 16-byte group; x: groups of a row, y: rows.
__global__ __launch_bounds__(256) void k_pad16(const uint16_t* __restrict__ src, int64_t ld_src,
                                               uint16_t* __restrict__ dst, int64_t ld_dst, int64_t rows,
                                               int64_t cols) {
  const int64_t c = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
  if (c >= ld_dst) return;
  for (int64_t r = blockIdx.y; r < rows; r += gridDim.y) {
    const uint16_t* s = src + r * ld_src + c;
    u32x4 v;
    if (c + 8 <= cols) {
      __builtin_memcpy(&v, s, 16);  // unaligned 16-byte load (gfx950 unaligned mode)
    } else {
      uint32_t h[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) h[e] = c + e < cols ? s[e] : 0u;
      v = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
    }
    __builtin_memcpy(dst + r * ld_dst + c, &v, 16);
  }
}

hipError_t launch_pad16(const uint16_t* src, int64_t ld_src, int64_t rows, int64_t cols, uint16_t* dst,
                        int64_t ld_dst, hipStream_t st) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  if (ld_src < cols || ld_dst < cols || (ld_dst & 7) != 0 || ((uintptr_t)dst & 15) != 0) return hipErrorInvalidValue;
  const int64_t gx = (ld_dst / 8 + 255) / 256;
  if (gx > (1LL << 31) - 1) return hipErrorInvalidValue;
  const dim3 grid((unsigned)gx, (unsigned)(rows < 4096 ? rows : 4096)), block(256);
  hipLaunchKernelGGL(k_pad16, grid, block, 0, st, src, ld_src, dst, ld_dst, rows, cols);
  return hipGetLastError();
}
#endif
}  // namespace ac
