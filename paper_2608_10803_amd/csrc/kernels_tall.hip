// gfx950 kernel for tall-skinny products, N <= 16 NT (NT = 1 or 2): the
// small-operand modules of Table 2 by orientation. A is the one large
// operand, so it is streamed from HBM exactly once at full cache-line width;
// B is read through its transposed copy B^T (N x K, rows padded to a
// multiple of 8), which a prologue writes into the workspace (T_pro of
// Eq. 7) and which stays in cache.
//
//   grid     ceil(M / BM) x P_k workgroups of 4 waves; workgroup (i, p) owns
//            rows BM i .. BM i + BM - 1 and K partition p (kper blocks of 64)
//   stage    one 64-deep k-block: A rows (BM x 128 bytes) and the matching
//            B^T rows (16 NT x 128 bytes), loaded straight into LDS
//            (buffer_load ... lds, chunks XOR-swizzled per row on the global
//            side); S stages, S - 1 of them in flight while one is multiplied
//            out (the Multi-Buffer module; Eq. 13 with a deeper pipeline)
//   compute  a wave owns BM / 4 rows: per 32-k half, BM / 64 A fragments and
//            NT B^T fragments (ds_read_b128 each, the same layout for both:
//            8 consecutive k of one row) into 16x16x32 MFMAs
//   output   the wave's rows x N columns of C (AddMM epilogue applied), or
//            an fp32 split-K partial that k_reduce sums (Eq. 11)
//
// Requirements (checked by the launcher): A row-major with 16-byte aligned
// rows (base 16-byte aligned, lda a multiple of 8 below 2^22), K a multiple
// of 8, B^T likewise. Rows past M, B^T rows past N and k past the
// partition's end are read as zeros through out-of-range buffer offsets.
//
// Register-load form (RG): A rows at any 2-byte alignment and any K >= 8.
// The same chunks go into the same LDS slots, fetched with 16-byte register
// loads (a chunk that crosses the row end as the 16 bytes ending there,
// shifted down; chunks past the partition as zeros) into a ring of S
// register sets, so that S blocks of loads are in flight; each step writes
// the oldest set into one of two LDS stages.
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

constexpr int TO_F32 = 0, TO_16 = 1, TO_PARTIAL = 2;  // C in fp32 or 16 bits, or a split-K partial

template <int NT, int BM, int S>
struct Tall {
  static constexpr int BM_ = BM, NT_ = NT;
  static constexpr int NB = 16 * NT;          // B^T rows (columns of C) of a stage
  static constexpr int RB = BM / 64;          // 16-row MFMA blocks of a wave
  static constexpr int A_BYTES = BM * 128;    // BM rows x 64 k
  static constexpr int B_BYTES = NB * 128;    // NB rows x 64 k
  static constexpr int ST_BYTES = A_BYTES + B_BYTES;
  static constexpr int NIA = A_BYTES / 4096;  // wave-wide A loads per wave and stage (8 rows each)
  static constexpr int B_LANES = B_BYTES / 64;  // lanes of each wave's one B^T load (32 or 64)
  static constexpr int LOADS = NIA + 1;         // load instructions per wave and stage
  static constexpr int WPE = 2 * S * ST_BYTES <= 160 * 1024 ? 2 : 1;  // workgroups per CU the LDS holds
  static_assert((NT == 1 || NT == 2) && BM % 64 == 0 && NIA >= 1, "tile");
  static_assert(S >= 2 && S <= 6 && (S - 2) * LOADS <= 63, "pipeline");
};

// Pipeline barrier: this wave's loads of the stage about to be read have
// landed (at most AHEAD later stages still in flight) and its LDS reads are
// done; then all waves meet, so every wave's loads of that stage have landed
// and no wave still reads the stage about to be reloaded.
template <int LOADS, int AHEAD>
__device__ __forceinline__ void tall_barrier() {
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(AHEAD * LOADS));
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Byte offset (from the workgroup's first row) of every chunk this lane
// loads, OOB_OFF for rows past M / N, and the chunk's k within the block.
template <class G>
struct TallAddr {
  const char* a;  // A + m0 * lda
  const char* bt;
  int32_t a_off[G::NIA], a_k[G::NIA];
  int32_t b_off, b_k;

  __device__ __forceinline__ void init(const GemmArgs& g, int64_t m0) {
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    a = reinterpret_cast<const char*>(g.A + m0 * g.lda);
    bt = reinterpret_cast<const char*>(g.B);
    const int64_t rows = g.M - m0;
#pragma unroll
    for (int q = 0; q < G::NIA; ++q) {
      const int row = (w * G::NIA + q) * 8 + (lane >> 3);
      const int c = (lane & 7) ^ swz_a<64>(row);  // the chunk that belongs at this lane's slot
      a_off[q] = row < rows ? (int32_t)(row * g.lda * 2) + c * 16 : OOB_OFF;
      a_k[q] = c * 8;
    }
    const int rb = w * (G::B_LANES / 8) + (lane >> 3);
    const int c = (lane & 7) ^ swz_a<64>(rb);
    b_off = rb < g.N ? (int32_t)(rb * g.ldb * 2) + c * 16 : OOB_OFF;
    b_k = c * 8;
  }

  // loads of the k-block starting at k0 (partition end kend) into a stage
  __device__ __forceinline__ void issue(char* stage, int64_t k0, int64_t kend) const {
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t kl = kend - k0;
    const int krem = kl <= 0 ? 0 : kl < 64 ? (int)kl : 64;  // uniform
    const __amdgpu_buffer_rsrc_t ra =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a) + k0 * 2, (short)0, (int)0x7FFFFFF0, (int)RSRC_WORD3);
    const __amdgpu_buffer_rsrc_t rb =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(bt) + k0 * 2, (short)0, (int)0x7FFFFFF0, (int)RSRC_WORD3);
#pragma unroll
    for (int q = 0; q < G::NIA; ++q)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(stage + (w * G::NIA + q) * 1024), 16,
                                               a_k[q] < krem ? a_off[q] : OOB_OFF, 0, 0, 0);
    if (G::B_LANES == 64 || lane < G::B_LANES)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void*)(stage + G::A_BYTES + w * (G::B_LANES * 16)), 16,
                                               b_k < krem ? b_off : OOB_OFF, 0, 0, 0);
  }
};

// ---- the register-load form
// Per lane: the byte offset of the (clamped) row of each A chunk it loads
// from the workgroup's first row, the chunk's k within the block, and the
// same for its one B^T chunk (rows past N, and lanes past the B^T tile,
// read zeros).
template <class G>
struct TallRegAddr {
  const uint16_t* a;   // A + m0 * lda
  const uint16_t* bt;  // B^T row of this lane's chunk (clamped)
  int64_t K, K8, kend;
  uint32_t a_off[G::NIA];
  int32_t a_c[G::NIA];
  int32_t b_c;
  bool b_on;

  __device__ __forceinline__ void init(const GemmArgs& g, int64_t m0, int64_t kend_) {
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    a = g.A + m0 * g.lda;
    K = g.K;
    K8 = (g.K + 7) / 8 * 8;
    kend = kend_;
#pragma unroll
    for (int q = 0; q < G::NIA; ++q) {
      const int row = (w * G::NIA + q) * 8 + (lane >> 3);
      a_off[q] = (uint32_t)((min(m0 + row, g.M - 1) - m0) * g.lda * 2);
      a_c[q] = ((lane & 7) ^ swz_a<64>(row)) * 8;
    }
    const int rb = w * (G::B_LANES / 8) + (lane >> 3);
    b_on = lane < G::B_LANES && rb < g.N;
    bt = g.B + min((int64_t)rb, g.N - 1) * g.ldb;
    b_c = ((lane & 7) ^ swz_a<64>(rb)) * 8;
  }
};

// One block of loads in registers: every lane always issues all G::LOADS
// loads (at clamped, valid addresses), so the per-wave load count of a
// block is fixed; `sh` holds, per chunk, the elements to drop (8 = all).
template <class G>
struct TallRegSet {
  static_assert(G::NIA + 1 <= 8, "shifts: 4 bits per chunk in 32 bits");
  u32x4 va[G::NIA], vb;
  uint32_t sh;

  __device__ __forceinline__ void issue(const TallRegAddr<G>& t, int64_t k0) {
    sh = 0;
#pragma unroll
    for (int q = 0; q < G::NIA; ++q) {
      const int64_t k = k0 + t.a_c[q], kk = min(k, t.K - 8);
      const uint32_t s = k >= t.kend ? 8u : (uint32_t)(k - kk);  // k - kk: elements past the row end
      va[q] = load16(reinterpret_cast<const uint16_t*>(reinterpret_cast<const char*>(t.a) + t.a_off[q]) + kk);
      sh |= s << (4 * q);
    }
    const int64_t k = k0 + t.b_c, kk = min(k, t.K8 - 8);  // B^T rows are zero-padded to K8
    vb = load16(t.bt + kk);
    sh |= (t.b_on && k < t.kend ? 0u : 8u) << (4 * G::NIA);
  }

  __device__ __forceinline__ void finish(char* stage) const {
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int q = 0; q < G::NIA; ++q)
      *reinterpret_cast<u32x4*>(stage + (w * G::NIA + q) * 1024 + lane * 16) = shift_down(va[q], (sh >> (4 * q)) & 15);
    if (G::B_LANES == 64 || lane < G::B_LANES)
      *reinterpret_cast<u32x4*>(stage + G::A_BYTES + w * (G::B_LANES * 16) + lane * 16) =
          shift_down(vb, (sh >> (4 * G::NIA)) & 15);
  }
};

// One stage multiplied out by one wave: two 32-k halves, RB x NT MFMAs each.
template <class G>
__device__ __forceinline__ void tall_compute(const char* stage, f32x4 (&acc)[G::RB][G::NT_]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int i16 = lane & 15, kg = lane >> 4;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int ch = 4 * h + kg;  // 8 consecutive k of the lane's k-group
    u32x4 a[G::RB], b[G::NT_];
#pragma unroll
    for (int r = 0; r < G::RB; ++r) {
      const int row = w * (G::BM_ / 4) + 16 * r + i16;
      a[r] = *reinterpret_cast<const u32x4*>(stage + row * 128 + ((ch ^ swz_a<64>(row)) << 4));
    }
#pragma unroll
    for (int n = 0; n < G::NT_; ++n) {
      const int rowb = 16 * n + i16;
      b[n] = *reinterpret_cast<const u32x4*>(stage + G::A_BYTES + rowb * 128 + ((ch ^ swz_a<64>(rowb)) << 4));
    }
#pragma unroll
    for (int r = 0; r < G::RB; ++r)
#pragma unroll
      for (int n = 0; n < G::NT_; ++n) acc[r][n] = mfma16(a[r], b[n], acc[r][n]);
  }
}

template <int NT, int BM, int S, int OUT, bool RG>
__device__ __forceinline__ void tall_kernel(const GemmArgs& g) {
  typedef Tall<NT, BM, S> G;
  // one array per stage, so that the wait before a read of one stage does
  // not also wait for the loads in flight into the others
  __shared__ __attribute__((aligned(1024))) char st0[G::ST_BYTES];
  __shared__ __attribute__((aligned(1024))) char st1[G::ST_BYTES];
  __shared__ __attribute__((aligned(1024))) char st2[G::ST_BYTES];
  __shared__ __attribute__((aligned(1024))) char st3[G::ST_BYTES];
  __shared__ __attribute__((aligned(1024))) char st4[G::ST_BYTES];
  __shared__ __attribute__((aligned(1024))) char st5[G::ST_BYTES];
  auto stage = [&](auto ic) -> char* {
    constexpr int I = decltype(ic)::value;
    return I == 0 ? st0 : I == 1 ? st1 : I == 2 ? st2 : I == 3 ? st3 : I == 4 ? st4 : st5;
  };

  const int64_t m0 = (int64_t)blockIdx.x * BM;
  const int split = blockIdx.y;
  const int64_t kbeg = min((int64_t)split * g.kper * 64, g.K);
  const int64_t kend = min(kbeg + (int64_t)g.kper * 64, g.K);
  const int nk = (int)((kend - kbeg + 63) / 64);

  f32x4 acc[G::RB][NT];
#pragma unroll
  for (int r = 0; r < G::RB; ++r)
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[r][n] = f32x4{0.f, 0.f, 0.f, 0.f};
  typedef std::integral_constant<int, 0> I0;
  typedef std::integral_constant<int, 1> I1;
  typedef std::integral_constant<int, 2> I2;
  typedef std::integral_constant<int, 3> I3;
  typedef std::integral_constant<int, 4> I4;
  typedef std::integral_constant<int, 5> I5;

  if constexpr (RG) {
    // register set I holds blocks I, I + S, ...; LDS stage I % 2 (S even)
    static_assert(S % 2 == 0, "register ring over two LDS stages");
    TallRegAddr<G> t;
    t.init(g, m0, kend);
    TallRegSet<G> rs[S];
#pragma unroll
    for (int b = 0; b < S; ++b) rs[b].issue(t, kbeg + (int64_t)b * 64);
    auto step = [&](auto ic, int kb) {
      constexpr int I = decltype(ic)::value;
      char* const st = I % 2 == 0 ? st0 : st1;
      rs[I].finish(st);  // the compiler waits for this set's loads only
      rs[I].issue(t, kbeg + (int64_t)(kb + S) * 64);
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");  // the stage is whole
      tall_compute<G>(st, acc);
    };
    int kb = 0;
    for (; kb + S <= nk; kb += S) {
      step(I0{}, kb);
      step(I1{}, kb + 1);
      step(I2{}, kb + 2);
      step(I3{}, kb + 3);
      if constexpr (S > 4) step(I4{}, kb + 4);
      if constexpr (S > 5) step(I5{}, kb + 5);
    }
    if (kb < nk) step(I0{}, kb);
    if (kb + 1 < nk) step(I1{}, kb + 1);
    if (kb + 2 < nk) step(I2{}, kb + 2);
    if constexpr (S > 4)
      if (kb + 3 < nk) step(I3{}, kb + 3);
    if constexpr (S > 5)
      if (kb + 4 < nk) step(I4{}, kb + 4);
  } else {
    TallAddr<G> t;
    t.init(g, m0);

    // stage I holds k-blocks I, I + S, ...; every step issues one stage of
    // loads (past the partition: all out of range), so S - 2 stages of loads
    // were issued after those of the block a step reads
  #pragma unroll
    for (int b = 0; b < S - 1; ++b) {
      char* const st = b == 0 ? st0 : b == 1 ? st1 : b == 2 ? st2 : b == 3 ? st3 : st4;
      t.issue(st, kbeg + (int64_t)b * 64, kend);
    }
    auto step = [&](auto ic, int kb) {
      constexpr int I = decltype(ic)::value;
      tall_barrier<G::LOADS, S - 2>();
      t.issue(stage(std::integral_constant<int, (I + S - 1) % S>{}), kbeg + (int64_t)(kb + S - 1) * 64, kend);
      tall_compute<G>(stage(ic), acc);
    };
    // whole groups of S blocks, then the remaining 0 .. S - 1
    int kb = 0;
    for (; kb + S <= nk; kb += S) {
      step(I0{}, kb);
      step(I1{}, kb + 1);
      if constexpr (S > 2) step(I2{}, kb + 2);
      if constexpr (S > 3) step(I3{}, kb + 3);
      if constexpr (S > 4) step(I4{}, kb + 4);
      if constexpr (S > 5) step(I5{}, kb + 5);
    }
    if (kb < nk) step(I0{}, kb);
    if constexpr (S > 2)
      if (kb + 1 < nk) step(I1{}, kb + 1);
    if constexpr (S > 3)
      if (kb + 2 < nk) step(I2{}, kb + 2);
    if constexpr (S > 4)
      if (kb + 3 < nk) step(I3{}, kb + 3);
    if constexpr (S > 5)
      if (kb + 4 < nk) step(I4{}, kb + 4);
  }

  // lane l, element e: row 4 (l / 16) + e of the 16-row block, column l % 16
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t rbase = m0 + w * (BM / 4) + 4 * (lane >> 4);
  float* part = g.ws + (size_t)split * (size_t)g.M * (size_t)g.ldw;
#pragma unroll
  for (int r = 0; r < G::RB; ++r)
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      const int64_t col = 16 * n + (lane & 15);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t row = rbase + 16 * r + e;
        if (row >= g.M || col >= g.N) continue;
        if constexpr (OUT == TO_PARTIAL) {
          part[row * g.ldw + col] = acc[r][n][e];
        } else {
          float v[1] = {acc[r][n][e]};
          epi_apply<OUT == TO_16, 1>(g, v, row, col, 1);
          store_c<OUT == TO_16>(g.C, row * g.ldc + col, v[0]);
        }
      }
    }
}

template <int NT, int BM, int S, int OUT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(Tall<NT, BM, S>::WPE, Tall<NT, BM, S>::WPE)))
void k_tall(GemmArgs g) {
  tall_kernel<NT, BM, S, OUT, false>(g);
}
template <int NT, int BM, int S, int OUT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(Tall<NT, BM, S>::WPE, Tall<NT, BM, S>::WPE)))
void k_tallu(GemmArgs g) {
  tall_kernel<NT, BM, S, OUT, true>(g);
}

constexpr bool tall_has_unal(int nt, int bm, int stages) {
  for (const TallCfg& t : kTallCfg)
    if (t.nt == nt && t.bm == bm && t.stages == stages) return t.unal != 0;
  return false;
}

template <int NT, int BM, int S>
hipError_t launch_tall(const Plan& p, const GemmArgs& g, hipStream_t st, bool o16) {
  const dim3 grid(p.grid_x, p.grid_y), block(256);
  if (p.unal) {
    if constexpr (tall_has_unal(NT, BM, S)) {
      if (p.pk > 1)
        hipLaunchKernelGGL((k_tallu<NT, BM, S, TO_PARTIAL>), grid, block, 0, st, g);
      else if (o16)
        hipLaunchKernelGGL((k_tallu<NT, BM, S, TO_16>), grid, block, 0, st, g);
      else
        hipLaunchKernelGGL((k_tallu<NT, BM, S, TO_F32>), grid, block, 0, st, g);
      return hipGetLastError();
    } else {
      return hipErrorInvalidValue;
    }
  }
  if (p.pk > 1)
    hipLaunchKernelGGL((k_tall<NT, BM, S, TO_PARTIAL>), grid, block, 0, st, g);
  else if (o16)
    hipLaunchKernelGGL((k_tall<NT, BM, S, TO_16>), grid, block, 0, st, g);
  else
    hipLaunchKernelGGL((k_tall<NT, BM, S, TO_F32>), grid, block, 0, st, g);
  return hipGetLastError();
}

template <int NT, int BM, int S>
int occ_tall() {
  int o = 1 << 20;
  const void* ks[6] = {reinterpret_cast<const void*>(k_tall<NT, BM, S, TO_F32>),
                       reinterpret_cast<const void*>(k_tall<NT, BM, S, TO_16>),
                       reinterpret_cast<const void*>(k_tall<NT, BM, S, TO_PARTIAL>), nullptr, nullptr, nullptr};
  if constexpr (tall_has_unal(NT, BM, S)) {  // the register-load form: one occupancy for both
    ks[3] = reinterpret_cast<const void*>(k_tallu<NT, BM, S, TO_F32>);
    ks[4] = reinterpret_cast<const void*>(k_tallu<NT, BM, S, TO_16>);
    ks[5] = reinterpret_cast<const void*>(k_tallu<NT, BM, S, TO_PARTIAL>);
  }
  for (const void* k : ks) {
    if (!k) continue;
    int a = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&a, k, 256, 0) != hipSuccess) a = 0;
    o = a < o ? a : o;
  }
  return o;
}

typedef hipError_t (*TallLaunchFn)(const Plan&, const GemmArgs&, hipStream_t, bool);
typedef int (*TallOccFn)();
#define TALL_CFGS(X) X(1, 128, 4), X(1, 128, 6), X(1, 256, 4), X(1, 64, 6), X(2, 128, 4), X(2, 256, 4)
#define TALL_L(a, b, c) &launch_tall<a, b, c>
#define TALL_O(a, b, c) &occ_tall<a, b, c>
#define TALL_C(a, b, c) {a, b, c, Tall<a, b, c>::WPE}
const TallLaunchFn kTallFns[] = {TALL_CFGS(TALL_L)};
const TallOccFn kTallOcc[] = {TALL_CFGS(TALL_O)};
constexpr int kTallCheck[][4] = {TALL_CFGS(TALL_C)};
constexpr bool tall_match() {
  for (int i = 0; i < N_TALL_CFG; ++i)
    if (kTallCheck[i][0] != kTallCfg[i].nt || kTallCheck[i][1] != kTallCfg[i].bm ||
        kTallCheck[i][2] != kTallCfg[i].stages || kTallCheck[i][3] != kTallCfg[i].occ)
      return false;
  return true;
}
static_assert(sizeof(kTallFns) / sizeof(kTallFns[0]) == N_TALL_CFG && tall_match(),
              "kernels (and their workgroups per CU) must follow kTallCfg");

}  // namespace

hipError_t launch_tall_main(const Plan& p, const GemmArgs& g, hipStream_t st) {
  if (p.family != FAM_TALL || p.cfg < 0 || p.cfg >= N_TALL_CFG || p.pk < 1) return hipErrorInvalidValue;
  if (g.N > 16 * kTallCfg[p.cfg].nt) return hipErrorInvalidValue;
  // direct loads: aligned operands; register loads: any A with K >= 8 (the
  // transposed copy of B is aligned either way)
  if (p.unal ? (!kTallCfg[p.cfg].unal || g.K < 8 || g.lda >= DL_MAX_LD || ((uintptr_t)g.B & 15) != 0 ||
                (g.ldb & 7) != 0 || g.ldb < (g.K + 7) / 8 * 8)
             : !ac::tall_operands_aligned(g))
    return hipErrorInvalidValue;
  if (p.pk > 1 && !g.ws) return hipErrorInvalidValue;
  return kTallFns[p.cfg](p, g, st, dtype_out16(p.s.dtype));
}

void query_occupancy_tall() {
  for (int i = 0; i < N_TALL_CFG; ++i) set_runtime_occupancy(FAM_TALL, i, kTallOcc[i]());
}

#if AC_INPUT_F16
}  // namespace f16
#else
bool tall_a_aligned(const void* A, int64_t lda, int64_t K) {
  return ((uintptr_t)A & 15) == 0 && (lda & 7) == 0 && (K & 7) == 0 && lda < DL_MAX_LD;
}
bool tall_operands_aligned(const GemmArgs& g) {
  return tall_a_aligned(g.A, g.lda, g.K) && ((uintptr_t)g.B & 15) == 0 && (g.ldb & 7) == 0 && g.ldb >= g.K &&
         g.ldb < DL_MAX_LD;
}
#endif
}  // namespace ac
