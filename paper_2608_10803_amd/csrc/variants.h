// The variant space: the kernel configurations compiled into the library.
// Shared by the planner (host arithmetic) and the launch registry.
#pragma once
#include <stdint.h>

namespace ac {

// Macro-tile configurations of the tile kernel (k granule BK = 64, LDS
// double buffered; 4 waves in a 2 x 2 grid, 8 waves in 2 x 4 for the 256-row
// tiles). ms = MFMA tile (32: 32x32x16, 16: 16x16x32). depth = k-blocks of
// global loads held in registers ahead of the LDS stage (1 or 2: two hide more
// latency on long K, one keeps more workgroups per CU). occ = workgroups per
// CU the planner assumes until the device reports the real figure. The first
// N_STREAMK_CFG configurations also have a stream-K kernel.
struct TileCfg {
  int bm, bn, ms, occ, depth;
};
constexpr int TILE_BK = 64;
constexpr TileCfg kTileCfg[] = {
    {256, 256, 32, 1, 1}, {256, 128, 32, 1, 1}, {128, 256, 32, 1, 2}, {128, 128, 32, 2, 1},
    {128, 64, 32, 2, 1},  {64, 128, 32, 2, 1},  {64, 64, 32, 4, 2},   {32, 32, 16, 8, 2},
    {128, 128, 32, 1, 2}, {128, 64, 32, 2, 2},  {64, 128, 32, 2, 2},
};
constexpr int N_TILE_CFG = sizeof(kTileCfg) / sizeof(kTileCfg[0]);
constexpr int N_STREAMK_CFG = 8;

inline int tile_lds_bytes(const TileCfg& t) { return 2 * (t.bm + t.bn) * TILE_BK * 2 + 16; }

// Tile configurations that also have a grouped kernel (the tile kernel over
// the groups of a grouped product).
constexpr bool kGroupedCfg[] = {false, true, true, true, true, true, true, false, true, false, false};
static_assert(sizeof(kGroupedCfg) / sizeof(kGroupedCfg[0]) == N_TILE_CFG, "grouped configurations");

// Tile configurations that also have a persistent kernel (one k-block of
// global loads ahead, carried across tiles): the depth-1 configurations.
constexpr bool kPersistCfg[] = {true, true, false, true, true, true, false, false, false, false, false};
static_assert(sizeof(kPersistCfg) / sizeof(kPersistCfg[0]) == N_TILE_CFG, "persistent configurations");
// Persistent configurations the class-fixed search offers (the open search
// and forced keys offer every one). The 256 x 256 one is left out: timed on
// the calibration shapes it was the fastest configuration on 3 of 49 (by at
// most 7 %), while the latency model prices it about 15 % low on write-bound
// shapes, where the two-per-CU direct-to-LDS tiles are faster.
constexpr bool kPersistSearch[] = {false, true, false, true, true, true, false, false, false, false, false};
static_assert(sizeof(kPersistSearch) / sizeof(kPersistSearch[0]) == N_TILE_CFG, "persistent search menu");

// Small-M Copy configurations: M <= 16*mt rows, wkw waves split the k-range
// of a workgroup (the others split its columns); a workgroup covers
// 128 * (4 / wkw) columns; k granule 32.
struct SkinnyMCfg {
  int mt, wkw, occ;
};
constexpr int SKINNY_BK = 32;
constexpr SkinnyMCfg kSkinnyMCfg[] = {{1, 1, 4}, {1, 4, 4}, {2, 1, 4}, {2, 4, 4}, {4, 1, 2}, {4, 4, 1}};
constexpr int N_SKINNY_M_CFG = sizeof(kSkinnyMCfg) / sizeof(kSkinnyMCfg[0]);
inline int skinny_m_cols(const SkinnyMCfg& c) { return 128 * (4 / c.wkw); }

// Small-N configurations: N <= 16*nt columns, a workgroup covers 64*rb rows
// and walks its K range in chunks of SKINNY_N_KMAX (the B^T slice it keeps
// in LDS).
struct SkinnyNCfg {
  int nt, rb, occ;
};
constexpr int SKINNY_N_KMAX = 512;
constexpr SkinnyNCfg kSkinnyNCfg[] = {{1, 2, 4}, {2, 2, 4}, {4, 2, 2}};
constexpr int N_SKINNY_N_CFG = sizeof(kSkinnyNCfg) / sizeof(kSkinnyNCfg[0]);
inline int skinny_n_rows(const SkinnyNCfg& c) { return 64 * c.rb; }

// Small-K configurations: K <= kmax; a thread computes a run of rows (a
// multiple of 4, at most SMALLK_MAX_ROWS) x 8 columns.
struct SmallKCfg {
  int kmax, occ;
};
constexpr SmallKCfg kSmallKCfg[] = {{8, 4}, {16, 2}};
constexpr int N_SMALLK_CFG = sizeof(kSmallKCfg) / sizeof(kSmallKCfg[0]);
constexpr int SMALLK_MAX_ROWS = 32;
// Wide rows (N >= SMALLK_WIN_MIN_N): a workgroup covers a band of rows and
// SMALLK_WIN_COLS columns (31 lines of bf16, 62 of fp32) and writes per row
// the line-aligned window of that width (k_smallk_win).
constexpr int SMALLK_WIN_COLS = 1984;
constexpr int SMALLK_WIN_MIN_N = 1024;

// Direct configurations: wk = 1: four waves cover 64 x 64 of C, each over
// all of K; wk = 4 or 16: that many waves split the K range of one 32 x 32
// block (a workgroup of 64 * wk threads).
struct DirectCfg {
  int wk, occ;
};
constexpr DirectCfg kDirectCfg[] = {{1, 4}, {4, 4}, {16, 1}};
constexpr int N_DIRECT_CFG = sizeof(kDirectCfg) / sizeof(kDirectCfg[0]);
inline int direct_tile(const DirectCfg& c) { return c.wk == 1 ? 64 : 32; }

// Direct-to-LDS tile configurations (family FAM_DL): BM x BN output tile, 4
// waves in a 2 x 2 grid (1 x 4 along N for tiles of at most 64 rows),
// k-blocks of bk (32 or 64; splits stay in units of
// TILE_BK), `stages` LDS stages (stages - 1 k-blocks of loads in flight);
// `occ` workgroups per CU (two for the configurations whose LDS stages and
// registers leave room for a second one). `unal`: the configuration also
// has a form that loads its operand tiles through registers at any
// alignment (K, N >= 8; VariantKey bit 13), in place of the padding
// prologue. When the caller's operands are not 16-byte aligned row by row,
// a plan of the direct-load form runs its register-load form if it has one,
// else `sibling`, the register-staged tile configuration of the same tiling
// (-1: none).
struct DlCfg {
  int bm, bn, bk, stages, sibling, occ, unal;
};
constexpr DlCfg kDlCfg[] = {{256, 256, 64, 2, 0, 1, 0}, {256, 128, 64, 3, 1, 1, 0}, {128, 256, 64, 3, 2, 1, 0},
                            {128, 128, 64, 3, 3, 1, 0}, {256, 256, 32, 4, 0, 1, 0}, {256, 256, 32, 5, 0, 1, 0},
                            {256, 128, 32, 4, 1, 1, 0}, {128, 256, 32, 4, 2, 1, 0}, {256, 128, 32, 2, 1, 2, 1},
                            {128, 128, 64, 2, 3, 2, 1}, {128, 128, 32, 2, 3, 2, 1},
                            // decode-style (few rows): 4 waves side by side along N, B streamed
                            // through 3-4 stages; no tile kernel has their tiling, so their
                            // register-load form is the fallback for unaligned operands
                            {32, 256, 64, 4, -1, 1, 1}, {64, 256, 64, 4, -1, 1, 1}, {32, 128, 64, 4, -1, 2, 1},
                            // a wide two-per-CU tile for write-bound shapes: 1 KB row segments of
                            // bf16 C per tile, so fewer lines shared with the neighbouring tiles
                            {64, 512, 32, 2, -1, 2, 1}};
constexpr bool dl_has_unal(int bm, int bn, int bk, int stages) {
  for (const DlCfg& d : kDlCfg)
    if (d.bm == bm && d.bn == bn && d.bk == bk && d.stages == stages) return d.unal != 0;
  return false;
}
constexpr int N_DL_CFG = sizeof(kDlCfg) / sizeof(kDlCfg[0]);

// leading dimensions of A and B the direct-to-LDS kernels address (elements)
constexpr int64_t DL_MAX_LD = 1LL << 22;

// Tall-skinny streaming configurations (N <= 16 nt): a workgroup owns bm
// rows of A and one K partition and streams them through `stages` LDS
// stages of 64 k (A: bm x 64, B^T: 16 nt x 64) with direct-to-LDS loads;
// occ workgroups per CU (what the LDS holds). unal: the configuration also
// has a register-load form (A rows at any alignment, K not a multiple of
// 8): `stages` blocks of loads in flight in registers, two LDS stages.
struct TallCfg {
  int nt, bm, stages, occ, unal;
};
constexpr TallCfg kTallCfg[] = {{1, 128, 4, 2, 1}, {1, 128, 6, 1, 1}, {1, 256, 4, 1, 0},
                                {1, 64, 6, 2, 1},  {2, 128, 4, 2, 1}, {2, 256, 4, 1, 0}};
constexpr int N_TALL_CFG = sizeof(kTallCfg) / sizeof(kTallCfg[0]);
inline int tall_lds_bytes(const TallCfg& t) { return t.stages * (t.bm + 16 * t.nt) * 128; }
inline int dl_lds_bytes(const DlCfg& d) { return d.stages * (d.bm + d.bn) * d.bk * 2; }

// 64-bit key of a configuration:
//   bits  0- 3 family, 4-11 config index, 12 swizzle, 13 operand loads
//   through registers (direct-to-LDS family), 16-35 P_k (or the stream-K
//   grid), 36-47 reserved, 48-51 dtype, 52-53 layouts.
inline uint64_t make_variant_key(int family, int cfg, int swizzle, int pk, int dtype, int layouts) {
  return (uint64_t)(family & 0xF) | ((uint64_t)(cfg & 0xFF) << 4) | ((uint64_t)(swizzle & 1) << 12) |
         ((uint64_t)(pk & 0xFFFFF) << 16) | ((uint64_t)(dtype & 0xF) << 48) | ((uint64_t)(layouts & 0x3) << 52);
}
inline int vk_family(uint64_t k) { return (int)(k & 0xF); }
inline int vk_cfg(uint64_t k) { return (int)((k >> 4) & 0xFF); }
inline int vk_swizzle(uint64_t k) { return (int)((k >> 12) & 1); }
inline int vk_unal(uint64_t k) { return (int)((k >> 13) & 1); }
inline int vk_pk(uint64_t k) { return (int)((k >> 16) & 0xFFFFF); }
inline int vk_dtype(uint64_t k) { return (int)((k >> 48) & 0xF); }
inline int vk_layouts(uint64_t k) { return (int)((k >> 52) & 0x3); }

}  // namespace ac
