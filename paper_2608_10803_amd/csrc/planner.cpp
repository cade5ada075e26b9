// Planner: taxonomy (Section 4.2 / 4.3), candidate enumeration and legality
// (Eq. 6), and the analytical latency model (Section 5.2, Eqs. 7-13) with
// MI355X stage costs.
#include "planner.h"

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdio>
#include <cstring>

namespace ac {

namespace {

std::atomic<int> g_occ[FAM_COUNT][16];

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Leading dimension of a split-K partial slice: N rounded up to 8 floats.
int64_t ldw8(int64_t n) { return (n + 7) / 8 * 8; }

int table_occ(int family, int cfg) {
  switch (family) {
    case FAM_TILE:
    case FAM_STREAMK:
    case FAM_GROUPED:
    case FAM_PERSIST:
    case FAM_BATCHED:
      return kTileCfg[cfg].occ;
    case FAM_SKINNY_M:
      return kSkinnyMCfg[cfg].occ;
    case FAM_SKINNY_N:
      return kSkinnyNCfg[cfg].occ;
    case FAM_SMALLK:
      return kSmallKCfg[cfg].occ;
    case FAM_DIRECT:
      return kDirectCfg[cfg].occ;
    case FAM_DL:
      return kDlCfg[cfg].occ;
    case FAM_TALL:
      return kTallCfg[cfg].occ;
    case FAM_DLSC:
      return kDlCfg[cfg & 0xF].occ;
  }
  return 1;
}

int out_bytes(int dtype) { return dtype_out_bytes(dtype); }

// Offsets of each family's configurations in the calibrated cost tables.
constexpr int IDX_TILE = 0;
constexpr int IDX_SKINNY_M = IDX_TILE + N_TILE_CFG;
constexpr int IDX_SKINNY_N = IDX_SKINNY_M + N_SKINNY_M_CFG;
constexpr int IDX_SMALLK = IDX_SKINNY_N + N_SKINNY_N_CFG;
constexpr int IDX_STREAMK = IDX_SMALLK + N_SMALLK_CFG;
constexpr int IDX_DIRECT = IDX_STREAMK + N_STREAMK_CFG;
constexpr int IDX_PERSIST = IDX_DIRECT + N_DIRECT_CFG;
constexpr int IDX_DL = IDX_PERSIST + N_TILE_CFG;
constexpr int IDX_DLU = IDX_DL + N_DL_CFG;  // the register-load forms, in configuration order
constexpr int n_dl_unal() {
  int n = 0;
  for (const DlCfg& d : kDlCfg) n += d.unal != 0;
  return n;
}
constexpr int IDX_TALL = IDX_DLU + n_dl_unal();
constexpr int IDX_TALLU = IDX_TALL + N_TALL_CFG;  // the tall kernels' register-load forms
constexpr int n_tall_unal() {
  int n = 0;
  for (const TallCfg& t : kTallCfg) n += t.unal != 0;
  return n;
}
static_assert(IDX_TALLU + n_tall_unal() <= AC_N_CFG, "calibrated cost tables");
int tallu_index(int cfg) {
  int n = 0;
  for (int i = 0; i < cfg; ++i) n += kTallCfg[i].unal != 0;
  return IDX_TALLU + n;
}
// cost slot of the register-load form of a direct-to-LDS configuration
int dlu_index(int cfg) {
  int n = 0;
  for (int i = 0; i < cfg; ++i) n += kDlCfg[i].unal != 0;
  return IDX_DLU + n;
}

// Tiles the taxonomy uses for its spatial predicate: the menu entries whose
// accumulation tile keeps the MFMA pipeline efficient (>= 128 x 128), largest
// first. Smaller menu tiles remain candidates of the search.
const int kBaseTiles[] = {0, 1, 2, 3};

// Work of one candidate, in the terms of Eqs. 8-13.
struct Work {
  int64_t units = 0;     // workgroups
  int occ = 1;           // workgroups per CU
  double L = 0;          // main-loop iterations of the longest workgroup
  double bytes_it = 0;   // global bytes loaded per iteration by one workgroup
  double mfma_it = 0;    // MFMA cycles per iteration on each SIMD
  double lds_it = 0;     // LDS bytes per iteration of one workgroup
  double out_unit = 0;   // bytes a workgroup writes at the end (tile or partial)
  double epi = 0;        // bytes read by the reduction kernel (Eq. 11), 0 = none
  double epi_out = 0;    // output bytes written by the reduction kernel
  double total_write = 0;// bytes written by the main kernel (output or partials)
  int idx = -1;          // configuration index of the calibrated costs
  double setup = 0;      // bytes a workgroup stages before its main loop
  double extra_lat = 0;  // further dependent load phases (memory latencies)
  double prefetch = 1;   // main-loop iterations of loads in flight
  double total_read = 0; // sum over workgroups of bytes read (Eq. 1 analogue)
  bool unaligned = false;
  bool swizzle = false;  // XCD-aware tile order (tile-family kernels)
};

// Eq. 8 with shared bandwidth: per-workgroup share of HBM (compulsory
// traffic) and of the CU's cache bandwidth (re-reads), and the Eq. 13
// double-buffered schedule, summed over rounds of resident workgroups (Eq. 7:
// the slowest CU decides; wave quantisation is the number of rounds).
double model_time(const Shape& s, const Work& w, const adaptcore_hw_t& hw, double compulsory) {
  if (w.units <= 0) return hw.t_launch;
  const double slots = (double)hw.n_cu * std::max(1, w.occ);
  const double eta = hw.hbm_eta * (w.unaligned ? hw.unaligned_eta : 1.0);
  const double agg_hbm = hw.hbm_bw * eta;
  // per-configuration efficiency of the output writes (calibrated; 1 if not)
  const double wr = (w.idx >= 0 && hw.cfg_wr[w.idx] > 0) ? hw.cfg_wr[w.idx] : 1.0;
  // fraction of loaded bytes that come from HBM (the rest hits L2 / MALL)
  double hbm_frac = 1.0;
  if (w.total_read > compulsory && w.total_read > 0) {
    const double hbm = compulsory + (w.total_read - compulsory) * (1.0 - hw.l2_hit);
    hbm_frac = std::min(1.0, hbm / w.total_read);
  }
  auto unit_time = [&](double conc) {
    const double per_cu = std::ceil(conc / hw.n_cu);
    const double bw_hbm = std::min(agg_hbm / conc, hw.l2_bw_cu / per_cu);
    const double bw_l2 = hw.l2_bw_cu / per_cu;
    double tM = w.bytes_it * hbm_frac / bw_hbm + w.bytes_it * (1.0 - hbm_frac) / bw_l2;
    tM = std::max(tM, hw.t_mem_latency / w.prefetch);
    // non-memory initiation interval (Eq. 9): calibrated per configuration,
    // else MFMA issue / LDS traffic; workgroups sharing a CU share it
    const double tP0 = (w.idx >= 0 && hw.cfg_iter[w.idx] > 0)
                           ? hw.cfg_iter[w.idx]
                           : std::max(w.mfma_it / (hw.clock_hz * hw.mfma_eta), w.lds_it / hw.lds_bw_cu);
    const double tP = tP0 * per_cu;
    // fixed cost of a workgroup: calibrated per configuration (prologue,
    // first-load latency and epilogue latency together), else the generic
    // workgroup cost plus one memory latency per dependent load phase
    const bool cal = w.idx >= 0 && hw.cfg_wg[w.idx] > 0;
    const double twg = cal ? hw.cfg_wg[w.idx] : hw.t_wg;
    const double lat = cal ? 0.0 : hw.t_mem_latency;
    const double t_fill = lat + tM + tP;  // first slice: load latency, load, compute
    const double t_drain = w.out_unit / (bw_hbm * wr);
    const double t_setup = (w.setup > 0 ? lat + w.setup / bw_l2 : 0.0) + w.extra_lat * hw.t_mem_latency;
    const double L = std::max(0.0, w.L);
    if (L == 0) return twg + t_setup + t_drain;
    const double t_loop = t_fill + (L - 1) * std::max(tM, tP);  // Eq. 13
    // With r >= 2 workgroups resident on a CU their phases drift apart: one
    // writes its output while another runs its main loop (the overlap that
    // Eq. 14's preloading gives consecutive tiles, here between co-resident
    // ones), so of the two phases only the longer one and a 1/r share of the
    // shorter one remain on the critical path. r = 1 is Eq. 13's sum.
    const double r = std::min(per_cu, (double)std::max(1, w.occ));
    return twg + t_setup + std::max(t_loop, t_drain) + std::min(t_loop, t_drain) / r;
  };
  const int64_t full = (int64_t)(w.units / slots);
  const double rem = (double)w.units - full * slots;
  double t_main = full * unit_time(slots);
  if (rem > 0) t_main += unit_time(rem);
  // aggregate HBM roof over the whole launch
  const double hbm_read = compulsory + (w.total_read - std::min(w.total_read, compulsory)) * (1.0 - hw.l2_hit);
  t_main = std::max(t_main, hbm_read / agg_hbm + w.total_write / (agg_hbm * wr));
  // the XCD-aware tile order's calibrated effect on the main kernel
  if (w.swizzle) t_main *= hw.swizzle_gain;
  // cross-workgroup reduction (Eq. 11) as a second kernel: one more launch, the
  // partials read back and the output written once
  double t_epi = 0;
  if (w.epi > 0) t_epi = hw.t_launch + hw.t_mem_latency + (w.epi + w.epi_out) / (hw.hbm_bw * hw.hbm_eta);
  (void)s;
  return hw.t_launch + t_main + t_epi;  // Eq. 7 (T_pro: added for column-major operands, add_prologue)
}

struct Ctx {
  const Shape& s;
  const adaptcore_hw_t& hw;
  double compulsory;
  int cbytes;
  bool unaligned;
  int cls = -1;  // the shape's class when the search is class-fixed (-1: every candidate)
};

// bytes of B (K x N, 16-bit)
inline double s_bytes_b(const Ctx& c) { return 2.0 * (double)c.s.K * (double)c.s.N; }

// The output tiling shared by the tile kernels and the direct-to-LDS
// kernels: bm x bn tiles, P_k partitions of whole 64-deep k-blocks, four
// waves in wm x wn, each wave's part of the tile in ms x ms MFMA blocks.
// Fills everything but the kernel's own identity (family, configuration,
// occupancy, cost slot, prefetch depth).
bool build_tiling(const Ctx& c, int bm, int bn, int wm, int wn, int ms, int pk_req, int swizzle, Plan* p, Work* w) {
  const Shape& s = c.s;
  const int64_t tm = cdiv(s.M, bm), tn = cdiv(s.N, bn);
  const int64_t kt = cdiv(s.K, TILE_BK);
  if (tm * tn > (1LL << 31) - 1) return false;
  int64_t pk = 1, kper = kt;
  if (pk_req > 1) {
    if (kt < 2) return false;
    kper = cdiv(kt, pk_req);
    pk = cdiv(kt, kper);
    if (pk != pk_req) return false;  // an equivalent key with the effective P_k exists
    if (pk > 65535) return false;
  }
  p->swizzle = swizzle;
  p->tile_m = bm;
  p->tile_n = bn;
  p->tile_k = TILE_BK;
  p->pm = (int)tm;
  p->pn = (int)tn;
  p->pk = (int)pk;
  p->kper = (int)std::max<int64_t>(kper, 0);
  p->grid_x = (int)(tm * tn);
  p->grid_y = (int)pk;
  if (pk > 1) {
    p->n_launch = 2;
    p->ws_bytes = pk * s.M * ldw8(s.N) * 4;
  }
  const int ks = ms == 32 ? 16 : 32, cyc = ms == 32 ? 32 : 16;
  const int TM = bm / wm / ms, TN = bn / wn / ms;
  const double bm_e = (double)s.M / tm, bn_e = (double)s.N / tn;
  w->units = tm * tn * pk;
  w->L = (double)kper;
  w->bytes_it = (bm_e + bn_e) * TILE_BK * 2;
  w->mfma_it = (double)TM * TN * (TILE_BK / ks) * cyc;
  w->lds_it = 4.0 * (TM + TN) * (TILE_BK / ks) * 64 * 16 + (bm + bn) * TILE_BK * 2;
  w->out_unit = bm_e * bn_e * (pk == 1 ? c.cbytes : 4);
  w->total_write = (double)s.M * s.N * (pk == 1 ? c.cbytes : 4.0 * pk);
  if (pk > 1) {
    w->epi = (double)pk * s.M * s.N * 4;
    w->epi_out = (double)s.M * s.N * c.cbytes;
  }
  w->total_read = (double)tm * tn * (bm_e + bn_e) * (double)s.K * 2;
  w->unaligned = c.unaligned;
  w->swizzle = swizzle != 0;
  return true;
}

bool build_tile(const Ctx& c, int cfg, int pk_req, int swizzle, Plan* p, Work* w) {
  const TileCfg& t = kTileCfg[cfg];
  if (tile_lds_bytes(t) > c.hw.lds_bytes) return false;
  if (!build_tiling(c, t.bm, t.bn, 2, 2, t.ms, pk_req, swizzle, p, w)) return false;
  p->family = FAM_TILE;
  p->cfg = cfg;
  w->occ = occupancy(FAM_TILE, cfg);
  w->idx = IDX_TILE + cfg;
  w->prefetch = t.depth;
  return true;
}

// Persistent tile kernel: min(tiles, CUs x occupancy) workgroups, each
// walking ceil(tiles / grid) tiles back to back (Eq. 13 over all of its
// k-blocks, the first block of every later tile fetched during the previous
// tile's epilogue).
bool build_persist(const Ctx& c, int cfg, int swizzle, Plan* p, Work* w) {
  if (cfg < 0 || cfg >= N_TILE_CFG || !kPersistCfg[cfg]) return false;
  const Shape& s = c.s;
  if (s.K < 8 || s.N < 8) return false;
  if (!build_tile(c, cfg, 1, swizzle, p, w)) return false;
  const int64_t ntiles = (int64_t)p->pm * p->pn;
  const int occ = occupancy(FAM_PERSIST, cfg);
  const int64_t grid = std::min<int64_t>(ntiles, (int64_t)c.hw.n_cu * std::max(1, occ));
  const int64_t per = cdiv(ntiles, grid);
  p->family = FAM_PERSIST;
  p->grid_x = (int)grid;
  p->grid_y = 1;
  w->units = grid;
  w->occ = occ;
  w->idx = IDX_PERSIST + cfg;
  w->L = (double)per * (double)p->kper;
  w->out_unit *= (double)per;
  return true;
}

// Direct-to-LDS tile kernel: the tile kernel's tiling and split counts with
// stages - 1 k-blocks of loads in flight (Eq. 13 with a deeper pipeline) and
// no register staging. Its operands need 16-byte aligned rows whose 16-byte
// chunks lie wholly inside or outside the matrix: a row-major A with K not a
// multiple of 8, or a row-major B with N not a multiple of 8, is first copied
// into a zero-padded form (the Padding module of Table 2, priced as T_pro by
// add_prologue). The caller's pointers and leading dimensions are checked at
// launch, which runs the register-staged sibling of the same tiling on the
// original operands when an operand that is not copied is not aligned.
bool build_dl(const Ctx& c, int cfg, int pk_req, int swizzle, int unal, Plan* p, Work* w) {
  if (cfg < 0 || cfg >= N_DL_CFG) return false;
  const DlCfg& d = kDlCfg[cfg];
  const Shape& s = c.s;
  if (s.K < 1) return false;
  // the register-load form: in place of the padding prologue, for row-major
  // operands whose rows are not whole 16-byte chunks
  if (unal && (!d.unal || s.layouts != AC_LAYOUT_ROW_ROW || s.K < 8 || s.N < 8 || ((s.K % 8) == 0 && (s.N % 8) == 0)))
    return false;
  if (dl_lds_bytes(d) > c.hw.lds_bytes) return false;
  // a tiling without a tile-family sibling falls back to its register-load
  // form on misaligned operands, which needs K, N >= 8
  if (d.sibling < 0 && (s.K < 8 || s.N < 8)) return false;
  // four waves in 2 x 2, or side by side along N for tiles of at most 64 rows
  const int wm = d.bm >= 128 ? 2 : 1;
  if (!build_tiling(c, d.bm, d.bn, wm, 4 / wm, 32, pk_req, swizzle, p, w)) return false;
  p->family = FAM_DL;
  p->cfg = cfg;
  p->unal = unal;
  w->occ = occupancy(FAM_DL, cfg);
  w->idx = unal ? dlu_index(cfg) : IDX_DL + cfg;
  // LDS traffic per iteration (one TILE_BK of k): the stage written once by
  // the loads, A read by every wave column and B by every wave row; the
  // pipeline holds (stages - 1) * bk of k in flight
  w->lds_it = (double)(d.bm * (1 + 4 / wm) + d.bn * (1 + wm)) * TILE_BK * 2;
  w->prefetch = (double)(d.stages - 1) * d.bk / TILE_BK;
  w->unaligned = false;
  return true;
}

// Off-chip accumulation (SingleCoreSplitK / HybridSplitK, Section 4.2): the
// super-tile of two vertically adjacent 256 x 256 tiles of DL configuration
// `key_cfg & 0xF` (0 or 4), whose fp32 accumulator (512 KiB) exceeds S_acc;
// the P_k k1-slices of K are taken by kc = 1 << (key_cfg >> 4) workgroups
// along K (kc = 1: SingleCoreSplitK), each flushing its tiles' partial sums
// after every slice (write volume 4 MN P_k + 2 MN, Eqs. 3 and 5), then the
// reduction kernel adds the slices. The tiling, partial workspace and padding
// prologue are those of the direct-to-LDS split-K plan with the same slices.
bool build_dlsc(const Ctx& c, int key_cfg, int pk_req, Plan* p, Work* w) {
  const int cfg = key_cfg & 0xF, kcl = key_cfg >> 4;
  if ((cfg != 0 && cfg != 4) || kcl > 10 || pk_req < 2) return false;
  const int kc = 1 << kcl;
  if (pk_req % kc != 0 || pk_req / kc < 2) return false;  // at least two slices per workgroup
  if (!build_dl(c, cfg, pk_req, 0, 0, p, w)) return false;
  const int64_t tm = p->pm, tn = p->pn, sup_m = cdiv(tm, 2);
  if (sup_m * tn > (1LL << 31) - 1) return false;
  const double per = (double)(pk_req / kc) * (tm > 1 ? 2.0 : 1.0);  // tiles x slices of a workgroup
  p->family = FAM_DLSC;
  p->cfg = key_cfg;
  p->grid_x = (int)(sup_m * tn);
  p->grid_y = kc;
  w->units = sup_m * tn * kc;
  w->L *= per;
  w->out_unit *= per;
  // B's slice is read from HBM once per super-tile (the lower tile finds it
  // in the L2), A's rows once per column of super-tiles
  w->total_read -= (double)(tm - sup_m) * (double)s_bytes_b(c);
  return true;
}

// Tall-skinny streaming kernel: A (row-major, K a multiple of 8) read once
// through the kernel's LDS pipeline, B through its transposed copy (the
// prologue add_prologue prices); ceil(M / bm) x P_k workgroups, each a run
// of 64-deep k-blocks.
bool build_tall(const Ctx& c, int cfg, int pk_req, int unal, Plan* p, Work* w) {
  if (cfg < 0 || cfg >= N_TALL_CFG) return false;
  const TallCfg& t = kTallCfg[cfg];
  const Shape& s = c.s;
  if (s.N > 16 * t.nt || (t.nt > 1 && s.N <= 16 * (t.nt / 2))) return false;  // the narrowest that fits
  if ((s.layouts & AC_LAYOUT_A_COL) || s.K < 8) return false;
  // direct loads need rows of whole 16-byte chunks; the register-load form
  // serves the other K
  if (unal ? (!t.unal || (s.K % 8) == 0) : (s.K % 8) != 0) return false;
  if (tall_lds_bytes(t) > c.hw.lds_bytes) return false;
  const int64_t rbk = cdiv(s.M, t.bm), kb = cdiv(s.K, TILE_BK);
  int64_t pk = 1, kper = kb;
  if (pk_req > 1) {
    if (kb < 2) return false;
    kper = cdiv(kb, pk_req);
    pk = cdiv(kb, kper);
    if (pk != pk_req || pk > 65535) return false;
  }
  if (rbk > (1LL << 31) - 1) return false;
  p->family = FAM_TALL;
  p->cfg = cfg;
  p->unal = unal;
  p->tile_m = t.bm;
  p->tile_n = 16 * t.nt;
  p->tile_k = TILE_BK;
  p->pm = (int)rbk;
  p->pn = 1;
  p->pk = (int)pk;
  p->kper = (int)kper;
  p->grid_x = (int)rbk;
  p->grid_y = (int)pk;
  if (pk > 1) {
    p->n_launch = 2;
    p->ws_bytes = pk * s.M * ldw8(s.N) * 4;
  }
  const double rows_e = (double)s.M / rbk;
  w->units = rbk * pk;
  w->occ = occupancy(FAM_TALL, cfg);
  w->idx = unal ? tallu_index(cfg) : IDX_TALL + cfg;
  w->L = (double)kper;
  w->bytes_it = (rows_e + s.N) * TILE_BK * 2;
  w->mfma_it = (double)(t.bm / 64) * t.nt * 2 * 16;  // two 32-k halves of 16x16x32 MFMAs per wave
  w->lds_it = (double)(t.bm + 16 * t.nt) * TILE_BK * 2 * 2;  // written by the loads, read once
  w->out_unit = rows_e * s.N * (pk == 1 ? c.cbytes : 4);
  w->total_write = (double)s.M * s.N * (pk == 1 ? c.cbytes : 4.0 * pk);
  if (pk > 1) {
    w->epi = (double)pk * s.M * s.N * 4;
    w->epi_out = (double)s.M * s.N * c.cbytes;
  }
  w->prefetch = t.stages - 1;
  w->total_read = 2.0 * s.M * s.K + 2.0 * s.K * s.N * rbk;  // B^T read by every row block (from cache)
  w->unaligned = false;
  return true;
}

bool build_skinny_m(const Ctx& c, int cfg, int pk_req, Plan* p, Work* w) {
  const SkinnyMCfg& k = kSkinnyMCfg[cfg];
  const Shape& s = c.s;
  if (s.M > 16 * k.mt) return false;
  if (k.mt > 1 && s.M <= 16 * (k.mt / 2)) return false;  // a smaller row count fits
  const int NB = skinny_m_cols(k);
  const int64_t cb = cdiv(s.N, NB);
  const int64_t kb = cdiv(s.K, SKINNY_BK);
  int64_t pk = 1, kper = kb;
  if (pk_req > 1) {
    if (kb < 2) return false;
    kper = cdiv(kb, pk_req);
    pk = cdiv(kb, kper);
    if (pk != pk_req || pk > 65535) return false;
  }
  if (cb > (1LL << 31) - 1) return false;
  p->family = FAM_SKINNY_M;
  p->cfg = cfg;
  p->tile_m = 16 * k.mt;
  p->tile_n = NB;
  p->tile_k = SKINNY_BK;
  p->pm = 1;
  p->pn = (int)cb;
  p->pk = (int)pk;
  p->kper = (int)kper;
  p->grid_x = (int)cb;
  p->grid_y = (int)pk;
  if (pk > 1) {
    p->n_launch = 2;
    p->ws_bytes = pk * s.M * ldw8(s.N) * 4;
  }
  const double nb_e = (double)s.N / cb;
  w->units = cb * pk;
  w->occ = occupancy(FAM_SKINNY_M, cfg);
  w->idx = IDX_SKINNY_M + cfg;
  w->L = std::ceil((double)kper / k.wkw);
  w->bytes_it = 32.0 * k.wkw * nb_e * 2 + 4.0 * k.mt * 16 * 32 * 2;
  w->mfma_it = 8.0 * k.mt * 16;
  w->lds_it = 0;
  w->out_unit = (double)s.M * nb_e * (pk == 1 ? c.cbytes : 4);
  w->total_write = (double)s.M * s.N * (pk == 1 ? c.cbytes : 4.0 * pk);
  if (pk > 1) {
    w->epi = (double)pk * s.M * s.N * 4;
    w->epi_out = (double)s.M * s.N * c.cbytes;
  }
  w->prefetch = 2;
  w->total_read = 2.0 * s.K * s.N + 2.0 * s.M * s.K * cb;
  w->unaligned = (s.N % 8) != 0;
  return true;
}

bool build_skinny_n(const Ctx& c, int cfg, int pk_req, Plan* p, Work* w) {
  const SkinnyNCfg& k = kSkinnyNCfg[cfg];
  const Shape& s = c.s;
  if (s.N > 16 * k.nt) return false;
  if (k.nt > 1 && s.N <= 16 * (k.nt / 2)) return false;
  const int R = skinny_n_rows(k);
  const int64_t rbk = cdiv(s.M, R);
  const int64_t kb = cdiv(s.K, SKINNY_BK);
  int64_t pk = 1, kper = kb;
  if (pk_req > 1) {
    if (kb < 2) return false;
    kper = cdiv(kb, pk_req);
    pk = cdiv(kb, kper);
    if (pk != pk_req || pk > 65535) return false;
  }
  if (rbk > (1LL << 31) - 1) return false;
  p->family = FAM_SKINNY_N;
  p->cfg = cfg;
  p->tile_m = R;
  p->tile_n = 16 * k.nt;
  p->tile_k = SKINNY_BK;
  p->pm = (int)rbk;
  p->pn = 1;
  p->pk = (int)pk;
  p->kper = (int)kper;
  p->grid_x = (int)rbk;
  p->grid_y = (int)pk;
  if (pk > 1) {
    p->n_launch = 2;
    p->ws_bytes = pk * s.M * ldw8(s.N) * 4;
  }
  const double rows_e = (double)s.M / rbk;
  w->units = rbk * pk;
  w->occ = occupancy(FAM_SKINNY_N, cfg);
  w->idx = IDX_SKINNY_N + cfg;
  w->L = (double)kper;
  w->bytes_it = rows_e * 32 * 2;
  w->mfma_it = (double)k.rb * k.nt * 16;
  w->lds_it = 64.0 * k.nt * 16 * 4;
  // B staged into LDS chunk by chunk (SKINNY_N_KMAX of K each); every chunk
  // after the first adds a dependent load phase
  w->setup = (double)kper * 32 * s.N * 2;
  w->extra_lat = (double)(cdiv(kper * SKINNY_BK, SKINNY_N_KMAX) - 1);
  w->out_unit = rows_e * s.N * (pk == 1 ? c.cbytes : 4);
  w->total_write = (double)s.M * s.N * (pk == 1 ? c.cbytes : 4.0 * pk);
  if (pk > 1) {
    w->epi = (double)pk * s.M * s.N * 4;
    w->epi_out = (double)s.M * s.N * c.cbytes;
  }
  w->prefetch = 2;
  w->total_read = 2.0 * s.M * s.K + 2.0 * s.K * s.N * rbk;
  w->unaligned = (s.K % 8) != 0;
  return true;
}

// Small problems: MFMA fragments straight from global memory, no LDS. One
// workgroup per 64 x 64 (wk = 1) or per 32 x 32 block of C with K split over
// its four waves (wk = 4).
bool build_direct(const Ctx& c, int cfg, int pk_req, Plan* p, Work* w) {
  const DirectCfg& d = kDirectCfg[cfg];
  const Shape& s = c.s;
  if (s.K < 1) return false;
  const int T = direct_tile(d);
  const int64_t tm = cdiv(s.M, T), tn = cdiv(s.N, T);
  if (tm * tn > (1LL << 31) - 1) return false;
  const int64_t kb = cdiv(s.K, 32);
  int64_t pk = 1, kper = kb;
  if (pk_req > 1) {
    if (kb < 2) return false;
    kper = cdiv(kb, pk_req);
    pk = cdiv(kb, kper);
    if (pk != pk_req || pk > 65535) return false;
  }
  const int64_t kb_wave = d.wk == 1 ? kper : cdiv(kper, d.wk);
  p->family = FAM_DIRECT;
  p->cfg = cfg;
  p->tile_m = T;
  p->tile_n = T;
  p->tile_k = 32;
  p->pm = (int)tm;
  p->pn = (int)tn;
  p->pk = (int)pk;
  p->kper = (int)kper;
  p->grid_x = (int)(tm * tn);
  p->grid_y = (int)pk;
  if (pk > 1) {
    p->n_launch = 2;
    p->ws_bytes = pk * s.M * ldw8(s.N) * 4;
  }
  w->units = tm * tn * pk;
  w->occ = occupancy(FAM_DIRECT, cfg);
  w->idx = IDX_DIRECT + cfg;
  // one iteration = one 32-k block of every wave: 16 B of A and 16 B of B
  // per lane and k-group
  const int waves = d.wk == 1 ? 4 : d.wk;
  w->L = (double)kb_wave;
  w->bytes_it = (double)waves * 64 * 32 * 2;
  w->mfma_it = 2.0 * 16;  // two 32x32x16 MFMAs of 16 cycles on each SIMD
  w->lds_it = 0;
  w->out_unit = (double)T * T * (pk == 1 ? c.cbytes : 4);
  w->total_write = (double)s.M * s.N * (pk == 1 ? c.cbytes : 4.0 * pk);
  if (pk > 1) {
    w->epi = (double)pk * s.M * s.N * 4;
    w->epi_out = (double)s.M * s.N * c.cbytes;
  }
  w->prefetch = 4;
  const double rows_read = (double)tn * s.M * s.K * 2, cols_read = (double)tm * s.K * s.N * 2;
  w->total_read = rows_read + cols_read;
  w->unaligned = (s.K % 8) != 0;
  return true;
}

// K <= 16: rank-K update with FMAs, one pass that writes C once.
bool build_smallk(const Ctx& c, int cfg, int pk_req, Plan* p, Work* w) {
  const SmallKCfg& k = kSmallKCfg[cfg];
  const Shape& s = c.s;
  if (pk_req != 1 || s.K > k.kmax || s.K < 1) return false;
  if (cfg > 0 && s.K <= kSmallKCfg[cfg - 1].kmax) return false;  // a smaller K bound fits
  const int64_t ncg = cdiv(s.N, 8);
  // rows per thread: the longest run (B read once per run) that still leaves
  // about 2048 threads per CU
  int64_t rpt = 4;
  while (rpt < SMALLK_MAX_ROWS && ncg * cdiv(s.M, 2 * rpt) >= (int64_t)c.hw.n_cu * 2048) rpt *= 2;
  const int64_t nrg = cdiv(s.M, rpt);
  // wide rows: line-aligned windows of SMALLK_WIN_COLS columns per band of
  // rpt rows (k_smallk_win); otherwise 256 consecutive threads of the
  // (row run, column group) order
  const bool win = s.N >= SMALLK_WIN_MIN_N && nrg <= 65535;
  const int64_t gx = win ? cdiv(s.N + 63, SMALLK_WIN_COLS) : cdiv(ncg * nrg, 256);
  const int64_t gy = win ? nrg : 1;
  if (gx > (1LL << 31) - 1) return false;
  p->family = FAM_SMALLK;
  p->cfg = cfg;
  p->tile_m = (int)rpt;
  p->tile_n = win ? SMALLK_WIN_COLS : 8;
  p->tile_k = k.kmax;
  p->pm = (int)std::min<int64_t>(nrg, (1LL << 31) - 1);
  p->pn = (int)(win ? gx : ncg);
  p->pk = 1;
  p->kper = (int)rpt;
  p->grid_x = (int)gx;
  p->grid_y = (int)gy;
  const int64_t wgs = gx * gy;
  w->units = wgs;
  w->occ = occupancy(FAM_SMALLK, cfg);
  w->idx = IDX_SMALLK + cfg;
  // one iteration = 4 rows of every thread: A rows (shared, cache hits)
  w->L = (double)rpt / 4;
  w->bytes_it = 256.0 * 4 * 16.0 * (k.kmax / 8);
  w->mfma_it = 4.0 * 8 * k.kmax * 4;  // FMA issue cycles of one wave (VALU, 4 cycles each)
  w->lds_it = 0;
  w->setup = 256.0 * s.K * 16.0;      // the B block of every thread
  w->out_unit = (win ? SMALLK_WIN_COLS : 256 * 8) * (double)rpt * c.cbytes;
  w->total_write = (double)s.M * s.N * c.cbytes;
  w->prefetch = 1;
  w->total_read = c.compulsory;  // re-reads of A rows and B rows stay in L1/L2
  w->unaligned = (s.N % 8) != 0 || (s.K % 8) != 0;
  return true;
}

// StreamK applied to the tile kernel: G persistent workgroups; the last
// partial wave of tiles (plus one full wave when there are at least two) is
// split evenly in MAC iterations, the rest runs data-parallel.
bool build_streamk(const Ctx& c, int cfg, Plan* p, Work* w) {
  const TileCfg& t = kTileCfg[cfg];
  const Shape& s = c.s;
  const int64_t tm = cdiv(s.M, t.bm), tn = cdiv(s.N, t.bn);
  const int64_t ntiles = tm * tn;
  const int64_t ipt = cdiv(s.K, TILE_BK);
  if (ntiles > (1LL << 30)) return false;
  const int64_t G = (int64_t)c.hw.n_cu * occupancy(FAM_STREAMK, cfg);
  int64_t sk;
  if (ipt < 2) {
    sk = 0;  // one k-block per tile: nothing to split, persistent data-parallel only
    if (ntiles <= G) return false;  // one tile per workgroup: the tile kernel itself
  } else if (ntiles >= G) {
    // a whole number of waves stays data-parallel (persistent workgroups,
    // each running its tiles back to back), otherwise the last partial wave
    // (plus one full wave when there are at least two) is split
    sk = ntiles % G;
    if (sk != 0 && ntiles >= 2 * G) sk += G;
  } else {
    sk = ntiles;
  }
  const int64_t ipw = sk > 0 ? cdiv(sk * ipt, G) : 0;
  const int64_t grid = std::min<int64_t>(G, std::max<int64_t>(cdiv(sk * ipt, ipw), 1));
  p->family = FAM_STREAMK;
  p->cfg = cfg;
  p->swizzle = 0;
  p->tile_m = t.bm;
  p->tile_n = t.bn;
  p->tile_k = TILE_BK;
  p->pm = (int)tm;
  p->pn = (int)tn;
  p->pk = (int)G;  // key field: the persistent grid
  p->kper = (int)ipt;
  (void)grid;
  p->grid_x = (int)G;
  p->grid_y = 1;
  p->iters_per_wg = (int)ipw;
  p->sk_tiles = (int)sk;
  p->ws_pk = sk > 0 ? (int)(cdiv(ipt, ipw) + 1) : 0;
  p->n_launch = sk > 0 ? 2 : 1;
  p->ws_bytes = (int64_t)sk * p->ws_pk * t.bm * t.bn * 4;
  const int ks = t.ms == 32 ? 16 : 32, cyc = t.ms == 32 ? 32 : 16;
  const int TM = t.bm / 2 / t.ms, TN = t.bn / 2 / t.ms;
  const double bm_e = (double)s.M / tm, bn_e = (double)s.N / tn;
  w->units = G;
  w->occ = occupancy(FAM_STREAMK, cfg);
  w->idx = IDX_STREAMK + cfg;
  w->L = (double)ipw + (double)cdiv(ntiles - sk, G) * ipt;
  w->bytes_it = (bm_e + bn_e) * TILE_BK * 2;
  w->mfma_it = (double)TM * TN * (TILE_BK / ks) * cyc;
  w->lds_it = 4.0 * (TM + TN) * (TILE_BK / ks) * 64 * 16 + (t.bm + t.bn) * TILE_BK * 2;
  w->out_unit = 2.0 * t.bm * t.bn * 4 + (double)((ntiles - sk) / G) * bm_e * bn_e * c.cbytes;
  w->total_write = (double)(ntiles - sk) * bm_e * bn_e * c.cbytes + (double)sk * 2 * t.bm * t.bn * 4;
  w->epi = (double)sk * 2 * t.bm * t.bn * 4;
  w->epi_out = (double)sk * bm_e * bn_e * c.cbytes;
  w->prefetch = 2;
  w->total_read = (double)ntiles * (bm_e + bn_e) * (double)s.K * 2;
  w->unaligned = c.unaligned;
  return true;
}

const int kSplits[] = {2, 3, 4, 5, 6, 8, 10, 12, 16, 20, 24, 32, 40, 48, 64, 80, 96, 128, 160, 192, 256, 384, 512, 768, 1024};

// Prologue of a plan with column-major operands: each one is copied into a
// row-major copy in the workspace (after the partials) by a transposing
// kernel, read and written once at the HBM rate: T_pro of Eq. 7, the same for
// every configuration of the shape except the small-M kernel, which reads a
// column-major B in place. Rows of the copies are padded to a multiple of 8
// elements (16-byte aligned rows for the main kernels).
void add_prologue(const Shape& s, const adaptcore_hw_t& hw, Plan* p) {
  p->ws_a_off = p->ws_b_off = -1;
  p->t_pro = 0;
  if (s.M == 0 || s.N == 0 || s.K == 0) return;
  auto copy = [&](int64_t rows, int64_t cols, int64_t* off) {
    *off = (p->ws_bytes + 255) / 256 * 256;
    p->ws_bytes = *off + rows * ldw8(cols) * 2;
    p->t_pro += hw.t_launch + 4.0 * (double)rows * (double)cols / (hw.hbm_bw * hw.hbm_eta);
    p->n_launch += 1;
  };
  if (s.layouts & AC_LAYOUT_A_COL) copy(s.M, s.K, &p->ws_a_off);
  // the padding prologue of the direct-to-LDS kernels: a row-major operand
  // whose rows are not whole 16-byte chunks is copied zero-padded
  else if ((p->family == FAM_DL || p->family == FAM_DLSC) && !p->unal && (s.K % 8) != 0) copy(s.M, s.K, &p->ws_a_off);
  // the small-M kernel reads a column-major B in place (its MFMA fragments
  // are runs of k), so only the other families copy B; the tall-skinny
  // kernel reads B's transposed copy (N x K, rows padded to 8) in any case
  if (p->family == FAM_TALL) copy(s.N, s.K, &p->ws_b_off);
  else if ((s.layouts & AC_LAYOUT_B_COL) && p->family != FAM_SKINNY_M) copy(s.K, s.N, &p->ws_b_off);
  else if (!(s.layouts & AC_LAYOUT_B_COL) && (p->family == FAM_DL || p->family == FAM_DLSC) && !p->unal && (s.N % 8) != 0)
    copy(s.K, s.N, &p->ws_b_off);
  p->predicted += p->t_pro;
}

bool finish(const Ctx& c, Plan* p, const Work& w) {
  p->s = c.s;
  p->predicted = model_time(c.s, w, c.hw, c.compulsory);
  p->variant_key = make_variant_key(p->family, p->cfg, p->swizzle, p->pk, c.s.dtype, (int)c.s.layouts) |
                   ((uint64_t)(p->unal & 1) << 13);
  add_prologue(c.s, c.hw, p);
  if (p->ws_bytes > ((int64_t)2 << 30)) return false;  // cap of the workspace: partials and operand copies
  return true;
}

// The grouped kernel for one tile configuration. Launch: an upper bound of
// the row tiles over any split of the rows into `groups` groups -- at most
// ne = min(groups, rows) groups hold rows, each adds at most one partial
// tile -- times the column tiles. Model: the counts are on the device, so
// the plan assumes the balanced split (ne groups of rows / ne rows) and
// prices it as ne independent products of that shape sharing the GPU.
bool build_grouped(const Shape& s, int64_t groups, const adaptcore_hw_t& hw, int cfg, int swizzle, Plan* p) {
  if (cfg < 0 || cfg >= N_TILE_CFG || !kGroupedCfg[cfg]) return false;
  const TileCfg& t = kTileCfg[cfg];
  if (tile_lds_bytes(t) > hw.lds_bytes) return false;
  const int64_t ne = std::min<int64_t>(groups, s.M);
  const int64_t slots = ne > 0 ? (s.M - ne) / t.bm + ne : 0;
  const int64_t tn = cdiv(s.N, t.bn);
  const int64_t threads = t.bm == 256 ? 512 : 256;
  if (slots * tn > (1LL << 31) - 1 || slots * tn * threads >= (1LL << 32)) return false;
  p->s = s;
  p->groups = groups;
  p->family = FAM_GROUPED;
  p->cfg = cfg;
  p->swizzle = swizzle;
  p->tile_m = t.bm;
  p->tile_n = t.bn;
  p->tile_k = TILE_BK;
  p->pm = (int)slots;
  p->pn = (int)tn;
  p->pk = 1;
  p->kper = (int)cdiv(s.K, TILE_BK);
  p->grid_x = (int)(slots * tn);
  p->grid_y = 1;
  p->n_launch = p->grid_x > 0 ? 1 : 0;
  p->ws_bytes = 0;
  p->variant_key = make_variant_key(FAM_GROUPED, cfg, swizzle, 1, s.dtype, (int)s.layouts);
  if (p->grid_x == 0) {
    p->predicted = 0;
    return true;
  }
  const Shape sg{cdiv(s.M, ne), s.N, s.K, s.dtype, s.layouts};
  const double compulsory = 2.0 * sg.M * sg.K + 2.0 * sg.K * sg.N;
  const bool unaligned = (s.K % 8) != 0 || (s.N % 8) != 0;
  const Ctx c{sg, hw, compulsory, out_bytes(s.dtype), unaligned};
  Plan one;
  Work w;
  if (!build_tile(c, cfg, 1, swizzle, &one, &w)) return false;
  w.units *= ne;
  w.total_read *= (double)ne;
  w.total_write *= (double)ne;
  p->predicted = model_time(sg, w, hw, compulsory * (double)ne);
  return true;
}

}  // namespace

adaptcore_hw_t default_hw() {
  adaptcore_hw_t h;
  std::memset(&h, 0, sizeof h);
  h.n_cu = 256;
  h.lds_bytes = 160 * 1024;
  h.s_acc_bytes = 256 * 1024;  // 4 waves x 64 lanes x 256 accumulation registers x 4 B
  h.clock_hz = 2.4e9;
  h.hbm_bw = 8.0e12;
  h.mfma_eta = 0.85;
  h.lds_bw_cu = 128.0 * 2.4e9;
  h.t_wg = 0.2e-6;
  h.search_open = 0;
  h.enable_streamk = 0;
  // Constants fitted to per-configuration timings of shapes of the
  // dynamic-shape, decode-style, small-MN large-K, write-bound,
  // compute-bound and tall-skinny workloads on one MI355X, each replay timed
  // after the caches were flushed (squared log error of the model over the
  // configurations within 1.5x of their shape's fastest, on a seeded half of
  // the 380 measured shapes; the other half is held out to check the
  // ranking), evaluated with the workgroups-per-CU that the device reports
  // for each kernel, which is what the planner uses at run time. The launch
  // cost is the measured per-kernel floor of back-to-back launches.
  h.t_launch = 1.9e-06;
  h.t_mem_latency = 1.217e-06;
  h.hbm_eta = 1;
  h.l2_bw_cu = 3.532e+10;
  h.unaligned_eta = 1;
  h.l2_hit = 5.128e-33;
  h.swizzle_gain = 0.9092;
  // per configuration (tile 0-10, skinny-M 11-16, skinny-N 17-19, small-K
  // 20-21, stream-K 22-29, direct 30-32, persistent 33-43, direct-to-LDS
  // 44-58 and their register-load forms 59-65, tall-skinny 66-71 and their
  // register-load forms 72-75; 0 = analytic estimate, no timing data)
  static const double kIter[AC_N_CFG] = {
      3.202e-06, 2.343e-06, 2.297e-06, 1.067e-06, 9.358e-14, 8.208e-07, 6.285e-07, 8.829e-07,
      1.211e-06, 9.358e-14, 9.358e-14, 1.614e-06, 1.54e-06, 1.247e-06, 1.319e-06, 6.514e-06,
      4.154e-06, 7.299e-07, 7.763e-07, 1.263e-06, 9.358e-14, 9.358e-14, 2.884e-07, 2.128e-06,
      7.211e-06, 2.01e-06, 1.913e-06, 1.532e-06, 5.342e-10, 7.214e-07, 9.015e-07, 8.849e-07,
      2.567e-07, 2.833e-06, 2.176e-06, 0, 9.358e-14, 9.358e-14, 9.358e-14, 0,
      0, 0, 0, 0, 2.071e-06, 1.291e-06, 1.309e-06, 3.586e-09,
      2.166e-06, 2.115e-06, 1.967e-07, 2.405e-07, 8.638e-07, 9.358e-14, 9.358e-14, 5.205e-10,
      2.543e-07, 5.736e-07, 9.358e-14, 1.737e-06, 9.358e-14, 9.358e-14, 1.743e-06, 1.775e-06,
      9.591e-07, 2.893e-06, 9.358e-14, 4.613e-13, 9.358e-14, 3.233e-07, 7.773e-07, 3.027e-13,
      7.236e-07, 7.183e-07, 4.089e-07, 8.225e-07, 0, 0, 0, 0,
      0, 0, 0, 0, 0, 0, 0, 0,
      0, 0, 0, 0, 0, 0, 0, 0};
  static const double kWg[AC_N_CFG] = {
      2.811e-06, 1.7e-06, 5.176e-06, 2.515e-06, 2.787e-06, 1.129e-06, 1.657e-06, 3.096e-07,
      3.643e-06, 3.33e-06, 3.424e-06, 2.401e-06, 2.429e-06, 6.703e-06, 7.161e-06, 9.791e-06,
      4.684e-05, 3.724e-06, 4.512e-06, 2.73e-05, 3.654e-06, 4.658e-06, 5.219e-05, 9.358e-14,
      1e-09, 9.358e-14, 4.328e-06, 9.358e-14, 1.326e-05, 3.699e-05, 9.358e-14, 9.358e-14,
      3.839e-08, 9.358e-14, 9.358e-14, 0, 9.358e-14, 9.358e-14, 2.042e-06, 0,
      0, 0, 0, 0, 7.505e-06, 4.832e-06, 5.656e-06, 3.277e-06,
      1.355e-05, 1.46e-05, 5.308e-06, 5.586e-06, 3.896e-06, 2.767e-06, 1.733e-06, 3.16e-06,
      2.93e-06, 1.309e-06, 3.332e-06, 2.74e-06, 4.905e-06, 2.538e-06, 5.649e-06, 8.669e-06,
      3.265e-06, 6.21e-07, 5.178e-06, 5.17e-06, 5.49e-06, 2.134e-06, 2.866e-06, 1.055e-05,
      4.831e-06, 5.186e-06, 3.93e-06, 2.981e-06, 0, 0, 0, 0,
      0, 0, 0, 0, 0, 0, 0, 0,
      0, 0, 0, 0, 0, 0, 0, 0};
  // achieved fraction of the streaming rate for the output writes (0: 1)
  static const double kWr[AC_N_CFG] = {
      1, 1, 1, 1, 0.6662, 1, 1, 1,
      1, 0.6619, 0.6664, 0.9999, 1, 0.9997, 1, 0.9999,
      0.9996, 1, 1, 0.9999, 0.9369, 1, 0.2732, 0.5701,
      0.281, 0.6292, 1, 0.6475, 0.05, 1, 1, 1,
      0.05, 0.5744, 0.6389, 0, 0.4172, 0.3277, 0.4146, 0,
      0, 0, 0, 0, 0.4079, 0.9994, 0.9991, 1,
      1, 1, 1, 1, 0.8409, 1, 0.8467, 1,
      1, 1, 0.8875, 0.6279, 0.9941, 0.8532, 0.9999, 1,
      1, 1, 1, 1, 0.1873, 1, 1, 1,
      0.1588, 1, 1, 0.1698, 0, 0, 0, 0,
      0, 0, 0, 0, 0, 0, 0, 0,
      0, 0, 0, 0, 0, 0, 0, 0};
  for (int i = 0; i < AC_N_CFG; ++i) {
    h.cfg_iter[i] = kIter[i];
    h.cfg_wg[i] = kWg[i];
    h.cfg_wr[i] = kWr[i];
  }
  return h;
}

void set_runtime_occupancy(int family, int cfg, int occ) {
  if (family >= 0 && family < FAM_COUNT && cfg >= 0 && cfg < 16) g_occ[family][cfg].store(occ);
}

int occupancy(int family, int cfg) {
  if (family == FAM_DLSC) {  // the direct-to-LDS configuration's kernel, looping
    family = FAM_DL;
    cfg &= 0xF;
  }
  const int o = g_occ[family][cfg].load(std::memory_order_relaxed);
  return o > 0 ? o : table_occ(family, cfg);
}

int classify_shape(const Shape& s, const adaptcore_hw_t& hw, int* base_cfg) {
  int base = -1;
  for (int cfg : kBaseTiles) {
    const TileCfg& t = kTileCfg[cfg];
    if (cdiv(s.M, t.bm) * cdiv(s.N, t.bn) >= hw.n_cu) {
      base = cfg;
      break;
    }
  }
  bool spatial = base >= 0;
  if (!spatial) base = kBaseTiles[sizeof(kBaseTiles) / sizeof(int) - 1];
  if (base_cfg) *base_cfg = base;
  const TileCfg& t = kTileCfg[base];
  const bool onchip = (int64_t)t.bm * t.bn * 4 <= hw.s_acc_bytes;
  if (spatial) return onchip ? AC_CLASS_COMMON : AC_CLASS_SINGLE_CORE_SPLITK;
  return onchip ? AC_CLASS_MULTI_CORE_SPLITK : AC_CLASS_HYBRID_SPLITK;
}

static void enumerate_all(const Ctx& c, std::vector<Plan>& out) {
  const Shape& s = c.s;
  auto add = [&](Plan& p, Work& w) {
    if (finish(c, &p, w)) out.push_back(p);
  };
  // tile kernel: every menu tile, P_k = 1 and the split counts
  for (int cfg = 0; cfg < N_TILE_CFG; ++cfg) {
    const TileCfg& t = kTileCfg[cfg];
    // a tile more than twice the matrix in a dimension only adds padding
    if ((t.bm > 2 * s.M && t.bm > 32) || (t.bn > 2 * s.N && t.bn > 32)) continue;
    for (int sw = 0; sw < 2; ++sw) {
      const int64_t ntiles = cdiv(s.M, t.bm) * cdiv(s.N, t.bn);
      if (sw == 1 && ntiles < 16) continue;  // nothing to reorder
      {
        Plan p;
        Work w;
        if (build_tile(c, cfg, 1, sw, &p, &w)) add(p, w);
      }
      for (int pk : kSplits) {
        if ((int64_t)pk * ntiles > 8LL * c.hw.n_cu * kTileCfg[cfg].occ) break;
        Plan p;
        Work w;
        if (build_tile(c, cfg, pk, sw, &p, &w)) add(p, w);
      }
    }
    if (c.hw.enable_streamk && cfg < N_STREAMK_CFG) {
      Plan p;
      Work w;
      if (build_streamk(c, cfg, &p, &w)) add(p, w);
    }
  }
  // persistent tile kernels: only where a workgroup gets more than one tile
  // (else they equal the tile kernel), and in the class-fixed search only
  // once their costs are calibrated
  for (int cfg = 0; cfg < N_TILE_CFG; ++cfg) {
    if (!kPersistCfg[cfg]) continue;
    const int idx = IDX_PERSIST + cfg;
    if (!c.hw.search_open && (!kPersistSearch[cfg] || !(c.hw.cfg_iter[idx] > 0 && c.hw.cfg_wg[idx] > 0))) continue;
    const TileCfg& t = kTileCfg[cfg];
    if ((t.bm > 2 * s.M && t.bm > 32) || (t.bn > 2 * s.N && t.bn > 32)) continue;
    const int64_t ntiles = cdiv(s.M, t.bm) * cdiv(s.N, t.bn);
    if (ntiles <= (int64_t)c.hw.n_cu * std::max(1, occupancy(FAM_PERSIST, cfg))) continue;
    for (int sw = 0; sw < 2; ++sw) {
      Plan p;
      Work w;
      if (build_persist(c, cfg, sw, &p, &w)) add(p, w);
    }
  }
  // direct-to-LDS tile kernels: in the class-fixed search only once their
  // costs are calibrated (each form separately)
  auto calibrated = [&](int idx) { return c.hw.search_open || (c.hw.cfg_iter[idx] > 0 && c.hw.cfg_wg[idx] > 0); };
  for (int cfg = 0; cfg < N_DL_CFG; ++cfg) {
    const DlCfg& d = kDlCfg[cfg];
    if (!calibrated(IDX_DL + cfg) && !(d.unal && calibrated(dlu_index(cfg)))) continue;
    // a tile more than twice the matrix only adds padding (the 32-row decode
    // tile is the smallest there is: any M)
    if ((d.bm > 2 * s.M && d.bm > 32) || d.bn > 2 * s.N) continue;
    for (int sw = 0; sw < 2; ++sw) {
      const int64_t ntiles = cdiv(s.M, d.bm) * cdiv(s.N, d.bn);
      if (sw == 1 && ntiles < 16) continue;
      for (int un = 0; un < 2; ++un) {
        if (!calibrated(un ? dlu_index(cfg) : IDX_DL + cfg)) continue;
        {
          Plan p;
          Work w;
          if (build_dl(c, cfg, 1, sw, un, &p, &w)) add(p, w);
        }
        for (int pk : kSplits) {
          if ((int64_t)pk * ntiles > 8LL * c.hw.n_cu * d.occ) break;
          Plan p;
          Work w;
          if (build_dl(c, cfg, pk, sw, un, &p, &w)) add(p, w);
        }
      }
    }
  }
  // off-chip accumulation: super-tiles of the 256 x 256 direct-to-LDS tiles
  // with 2 to 32 k1-slices, taken by 1 (SingleCoreSplitK) or more
  // (HybridSplitK) workgroups along K; the class-fixed search keeps them for
  // the two off-chip templates only (enumerate)
  const bool offchip = c.hw.search_open || c.cls < 0 || c.cls == AC_CLASS_SINGLE_CORE_SPLITK ||
                       c.cls == AC_CLASS_HYBRID_SPLITK;
  for (int cfg : {0, 4}) {
    const DlCfg& d = kDlCfg[cfg];
    if (!offchip || !calibrated(IDX_DL + cfg) || d.bm > 2 * s.M || d.bn > 2 * s.N) continue;
    const int64_t kt = cdiv(s.K, TILE_BK), sup = cdiv(cdiv(s.M, d.bm), 2) * cdiv(s.N, d.bn);
    for (int pk : kSplits) {
      if (pk > 32 || pk > kt) break;
      for (int kcl = 0; (1 << kcl) <= pk / 2; ++kcl) {
        if (pk % (1 << kcl) != 0) continue;
        if ((int64_t)(1 << kcl) * sup > 8LL * c.hw.n_cu * d.occ) break;
        Plan p;
        Work w;
        if (build_dlsc(c, cfg | (kcl << 4), pk, &p, &w)) add(p, w);
      }
    }
  }
  // tall-skinny streaming kernels: in the class-fixed search once calibrated
  for (int cfg = 0; cfg < N_TALL_CFG; ++cfg) {
    const int un = (s.K % 8) != 0;  // the form this K takes
    if (un && !kTallCfg[cfg].unal) continue;
    if (!calibrated(un ? tallu_index(cfg) : IDX_TALL + cfg)) continue;
    const int64_t rbk = cdiv(s.M, kTallCfg[cfg].bm);
    {
      Plan p;
      Work w;
      if (build_tall(c, cfg, 1, un, &p, &w)) add(p, w);
    }
    for (int pk : kSplits) {
      if ((int64_t)pk * rbk > 8LL * c.hw.n_cu * kTallCfg[cfg].occ) break;
      Plan p;
      Work w;
      if (build_tall(c, cfg, pk, un, &p, &w)) add(p, w);
    }
  }
  for (int cfg = 0; cfg < N_SKINNY_M_CFG; ++cfg) {
    const int64_t cb = cdiv(s.N, skinny_m_cols(kSkinnyMCfg[cfg]));
    {
      Plan p;
      Work w;
      if (build_skinny_m(c, cfg, 1, &p, &w)) add(p, w);
    }
    for (int pk : kSplits) {
      if ((int64_t)pk * cb > 8LL * c.hw.n_cu * kSkinnyMCfg[cfg].occ) break;
      Plan p;
      Work w;
      if (build_skinny_m(c, cfg, pk, &p, &w)) add(p, w);
    }
  }
  for (int cfg = 0; cfg < N_SKINNY_N_CFG; ++cfg) {
    const int64_t rb = cdiv(s.M, skinny_n_rows(kSkinnyNCfg[cfg]));
    {
      Plan p;
      Work w;
      if (build_skinny_n(c, cfg, 1, &p, &w)) add(p, w);
    }
    for (int pk : kSplits) {
      if ((int64_t)pk * rb > 8LL * c.hw.n_cu * kSkinnyNCfg[cfg].occ) break;
      Plan p;
      Work w;
      if (build_skinny_n(c, cfg, pk, &p, &w)) add(p, w);
    }
  }
  for (int cfg = 0; cfg < N_SMALLK_CFG; ++cfg) {
    Plan p;
    Work w;
    if (build_smallk(c, cfg, 1, &p, &w)) add(p, w);
  }
  for (int cfg = 0; cfg < N_DIRECT_CFG; ++cfg) {
    const int T = direct_tile(kDirectCfg[cfg]);
    const int64_t tiles = cdiv(s.M, T) * cdiv(s.N, T);
    {
      Plan p;
      Work w;
      if (build_direct(c, cfg, 1, &p, &w)) add(p, w);
    }
    for (int pk : kSplits) {
      if ((int64_t)pk * tiles > 8LL * c.hw.n_cu * kDirectCfg[cfg].occ) break;
      Plan p;
      Work w;
      if (build_direct(c, cfg, pk, &p, &w)) add(p, w);
    }
  }
}

std::vector<Plan> enumerate(const Shape& s, const adaptcore_hw_t& hw, int* cls_out) {
  int base = 0;
  const int cls = classify_shape(s, hw, &base);
  if (cls_out) *cls_out = cls;
  const double compulsory = 2.0 * s.M * s.K + 2.0 * s.K * s.N;
  const bool unaligned = (s.K % 8) != 0 || (s.N % 8) != 0;
  Ctx c{s, hw, compulsory, out_bytes(s.dtype), unaligned, cls};
  std::vector<Plan> all;
  enumerate_all(c, all);
  std::vector<Plan> sel;
  if (hw.search_open) {
    sel = all;
  } else {
    // Eq. 6: the search stays inside the template the taxonomy chose. The
    // spatially saturated templates keep k = K (no K split, no stream-K); the
    // K-parallel templates search the split count P_k, whose degenerate value
    // P_k = 1 is kept because a small problem can lose more to the reduction
    // than it gains from the idle cores.
    //
    // The spatial predicate P_m * P_n >= N_core is a property of the tiling
    // (Section 4.2), so it is applied to each candidate's own tile: a tile
    // that leaves CUs idle on this shape belongs to a K-parallel template and
    // keeps its split variants even when the taxonomy's base tile fills the
    // GPU.
    const bool ksplit = cls == AC_CLASS_MULTI_CORE_SPLITK || cls == AC_CLASS_HYBRID_SPLITK;
    const bool offchip = cls == AC_CLASS_SINGLE_CORE_SPLITK || cls == AC_CLASS_HYBRID_SPLITK;
    for (const Plan& p : all) {
      // off-chip accumulation only in its templates; its K is split across
      // workgroups only in HybridSplitK (SingleCoreSplitK keeps k = K)
      if (p.family == FAM_DLSC && !offchip) continue;
      const bool pk_split = p.family == FAM_STREAMK ? true : p.family == FAM_DLSC ? p.grid_y > 1 : p.pk > 1;
      const bool tile_idle = p.tile_m > 0 && p.tile_n > 0 &&
                             cdiv(s.M, p.tile_m) * cdiv(s.N, p.tile_n) < (int64_t)hw.n_cu;
      if (ksplit || tile_idle || !pk_split) sel.push_back(p);
    }
    if (sel.empty()) sel = all;
  }
  for (Plan& p : sel) p.cls = cls;
  std::stable_sort(sel.begin(), sel.end(), [](const Plan& a, const Plan& b) {
    if (a.predicted != b.predicted) return a.predicted < b.predicted;
    return a.variant_key < b.variant_key;
  });
  for (Plan& p : sel) p.n_candidates = (int)sel.size();
  return sel;
}

bool plan_for_key(const Shape& s, const adaptcore_hw_t& hw, uint64_t key, Plan* out) {
  if (vk_dtype(key) != s.dtype || vk_layouts(key) != (int)s.layouts) return false;
  int base = 0;
  const int cls = classify_shape(s, hw, &base);
  const double compulsory = 2.0 * s.M * s.K + 2.0 * s.K * s.N;
  const bool unaligned = (s.K % 8) != 0 || (s.N % 8) != 0;
  Ctx c{s, hw, compulsory, out_bytes(s.dtype), unaligned};
  const int fam = vk_family(key), cfg = vk_cfg(key), pk = vk_pk(key), sw = vk_swizzle(key);
  Plan p;
  Work w;
  bool ok = false;
  switch (fam) {
    case FAM_TILE:
      ok = cfg < N_TILE_CFG && pk >= 1 && build_tile(c, cfg, pk, sw, &p, &w);
      break;
    case FAM_SKINNY_M:
      ok = sw == 0 && cfg < N_SKINNY_M_CFG && pk >= 1 && build_skinny_m(c, cfg, pk, &p, &w);
      break;
    case FAM_SKINNY_N:
      ok = sw == 0 && cfg < N_SKINNY_N_CFG && pk >= 1 && build_skinny_n(c, cfg, pk, &p, &w);
      break;
    case FAM_STREAMK:
      ok = sw == 0 && cfg < N_STREAMK_CFG && build_streamk(c, cfg, &p, &w) && p.pk == pk;
      break;
    case FAM_SMALLK:
      ok = sw == 0 && cfg < N_SMALLK_CFG && build_smallk(c, cfg, pk, &p, &w);
      break;
    case FAM_DIRECT:
      ok = sw == 0 && cfg < N_DIRECT_CFG && build_direct(c, cfg, pk, &p, &w);
      break;
    case FAM_PERSIST:
      ok = pk == 1 && build_persist(c, cfg, sw, &p, &w);
      break;
    case FAM_DL:
      ok = cfg < N_DL_CFG && pk >= 1 && build_dl(c, cfg, pk, sw, vk_unal(key), &p, &w);
      break;
    case FAM_TALL:
      ok = sw == 0 && pk >= 1 && build_tall(c, cfg, pk, vk_unal(key), &p, &w);
      break;
    case FAM_DLSC:
      ok = sw == 0 && vk_unal(key) == 0 && build_dlsc(c, cfg, pk, &p, &w);
      break;
  }
  if (!ok || !finish(c, &p, w)) return false;
  if (p.variant_key != key) return false;
  p.cls = cls;
  p.n_candidates = 1;
  *out = p;
  return true;
}

// The grouped kernel over a strided batch: every group has the shape s, so
// the grid is exact (batch x row tiles x column tiles) and the model prices
// `batch` independent products of shape s sharing the GPU.
bool build_batched(const Shape& s, int64_t batch, const adaptcore_hw_t& hw, int cfg, int swizzle, Plan* p) {
  if (cfg < 0 || cfg >= N_TILE_CFG || !kGroupedCfg[cfg]) return false;
  const TileCfg& t = kTileCfg[cfg];
  if (tile_lds_bytes(t) > hw.lds_bytes) return false;
  const int64_t tpg = cdiv(s.M, t.bm), tn = cdiv(s.N, t.bn);
  const int64_t slots = batch * tpg;
  const int64_t threads = t.bm == 256 ? 512 : 256;
  if (slots * tn > (1LL << 31) - 1 || slots * tn * threads >= (1LL << 32)) return false;
  p->s = s;
  p->groups = batch;
  p->family = FAM_BATCHED;
  p->cfg = cfg;
  p->swizzle = swizzle;
  p->tile_m = t.bm;
  p->tile_n = t.bn;
  p->tile_k = TILE_BK;
  p->pm = (int)slots;
  p->pn = (int)tn;
  p->pk = 1;
  p->kper = (int)cdiv(s.K, TILE_BK);
  p->grid_x = (int)(slots * tn);
  p->grid_y = 1;
  p->n_launch = p->grid_x > 0 ? 1 : 0;
  p->ws_bytes = 0;
  p->variant_key = make_variant_key(FAM_BATCHED, cfg, swizzle, 1, s.dtype, (int)s.layouts);
  if (p->grid_x == 0) {
    p->predicted = 0;
    return true;
  }
  const double compulsory = 2.0 * s.M * s.K + 2.0 * s.K * s.N;
  const bool unaligned = (s.K % 8) != 0 || (s.N % 8) != 0;
  const Ctx c{s, hw, compulsory, out_bytes(s.dtype), unaligned};
  Plan one;
  Work w;
  if (!build_tile(c, cfg, 1, swizzle, &one, &w)) return false;
  w.units *= batch;
  w.total_read *= (double)batch;
  w.total_write *= (double)batch;
  p->predicted = model_time(s, w, hw, compulsory * (double)batch);
  return true;
}

bool plan_grouped(const Shape& s, int64_t groups, const adaptcore_hw_t& hw, Plan* out) {
  bool found = false;
  int n = 0;
  for (int cfg = 0; cfg < N_TILE_CFG; ++cfg) {
    Plan p;
    if (!build_grouped(s, groups, hw, cfg, 1, &p)) continue;
    ++n;
    if (!found || p.predicted < out->predicted) {
      *out = p;
      found = true;
    }
  }
  if (found) {
    int base = 0;
    out->n_candidates = n;
    out->cls = classify_shape(s, hw, &base);
  }
  return found;
}

bool grouped_for_key(const Shape& s, int64_t groups, const adaptcore_hw_t& hw, uint64_t key, Plan* out) {
  if (vk_family(key) != FAM_GROUPED || vk_pk(key) != 1 || vk_dtype(key) != s.dtype ||
      vk_layouts(key) != (int)s.layouts)
    return false;
  Plan p;
  if (!build_grouped(s, groups, hw, vk_cfg(key), vk_swizzle(key), &p) || p.variant_key != key) return false;
  int base = 0;
  p.n_candidates = 1;
  p.cls = classify_shape(s, hw, &base);
  *out = p;
  return true;
}

bool plan_batched(const Shape& s, int64_t batch, const adaptcore_hw_t& hw, Plan* out) {
  bool found = false;
  int n = 0;
  for (int cfg = 0; cfg < N_TILE_CFG; ++cfg) {
    Plan p;
    if (!build_batched(s, batch, hw, cfg, 1, &p)) continue;
    ++n;
    if (!found || p.predicted < out->predicted) {
      *out = p;
      found = true;
    }
  }
  if (found) {
    int base = 0;
    out->n_candidates = n;
    out->cls = classify_shape(s, hw, &base);
  }
  return found;
}

bool batched_for_key(const Shape& s, int64_t batch, const adaptcore_hw_t& hw, uint64_t key, Plan* out) {
  if (vk_family(key) != FAM_BATCHED || vk_pk(key) != 1 || vk_dtype(key) != s.dtype ||
      vk_layouts(key) != (int)s.layouts)
    return false;
  Plan p;
  if (!build_batched(s, batch, hw, vk_cfg(key), vk_swizzle(key), &p) || p.variant_key != key) return false;
  int base = 0;
  p.n_candidates = 1;
  p.cls = classify_shape(s, hw, &base);
  *out = p;
  return true;
}

static std::string kernel_names_fmt(const Plan& p);

std::string kernel_names(const Plan& p) {
  // the fp16-input kernels live in the nested namespace f16
  std::string r = kernel_names_fmt(p);
  if (dtype_f16_input(p.s.dtype) && !r.empty()) {
    std::string out = "f16::";
    for (char ch : r) {
      out += ch;
      if (ch == ';') out += "f16::";
    }
    r = out;
  }
  // the prologue (one copy kernel per copied operand: a transpose for a
  // column-major operand, the padding copy otherwise) runs first
  // (the tall-skinny kernel's copy of B is B^T: a transpose of a row-major B)
  const bool b_tr = ((p.s.layouts & AC_LAYOUT_B_COL) != 0) != (p.family == FAM_TALL);
  if (p.ws_b_off >= 0) r = std::string(b_tr ? "k_transpose16;" : "k_pad16;") + r;
  if (p.ws_a_off >= 0) r = std::string((p.s.layouts & AC_LAYOUT_A_COL) ? "k_transpose16;" : "k_pad16;") + r;
  return r;
}

static std::string kernel_names_fmt(const Plan& p) {
  const int obf = dtype_out16(p.s.dtype);
  const char* b = obf ? "true" : "false";
  char buf[160];
  switch (p.family) {
    case FAM_TILE: {
      const TileCfg& t = kTileCfg[p.cfg];
      std::snprintf(buf, sizeof buf, "k_tile<%d, %d, %d, %d, %d>", t.bm, t.bn, t.ms, p.pk > 1 ? 2 : obf, t.depth);
      std::string r(buf);
      if (p.pk > 1) r += std::string(";k_reduce<") + b + ">";
      return r;
    }
    case FAM_STREAMK: {
      const TileCfg& t = kTileCfg[p.cfg];
      std::snprintf(buf, sizeof buf, "k_streamk<%d, %d, %d, %s>", t.bm, t.bn, t.ms, b);
      std::string r(buf);
      if (p.sk_tiles > 0) r += std::string(";k_sk_fixup<") + b + ">";
      return r;
    }
    case FAM_SKINNY_M: {
      const SkinnyMCfg& k = kSkinnyMCfg[p.cfg];
      const bool bt = (p.s.layouts & AC_LAYOUT_B_COL) && p.ws_b_off < 0;
      std::snprintf(buf, sizeof buf, "k_skinny_m%s<%d, %d, %s>", bt ? "_bt" : "", k.mt, k.wkw, b);
      std::string r(buf);
      if (p.pk > 1) r += std::string(";k_reduce<") + b + ">";
      return r;
    }
    case FAM_SKINNY_N: {
      const SkinnyNCfg& k = kSkinnyNCfg[p.cfg];
      std::snprintf(buf, sizeof buf, "k_skinny_n<%d, %d, %s>", k.nt, k.rb, b);
      std::string r(buf);
      if (p.pk > 1) r += std::string(";k_reduce<") + b + ">";
      return r;
    }
    case FAM_SMALLK:
      std::snprintf(buf, sizeof buf, p.tile_n == SMALLK_WIN_COLS ? "k_smallk_win<%d, %s>" : "k_smallk<%d, %s>",
                    kSmallKCfg[p.cfg].kmax, b);
      return buf;
    case FAM_PERSIST: {
      const TileCfg& t = kTileCfg[p.cfg];
      std::snprintf(buf, sizeof buf, "k_tile_pp<%d, %d, %d, %s>", t.bm, t.bn, t.ms, b);
      return buf;
    }
    case FAM_GROUPED:
    case FAM_BATCHED: {
      const TileCfg& t = kTileCfg[p.cfg];
      std::snprintf(buf, sizeof buf, "k_grouped<%d, %d, %d, %d, %d>", t.bm, t.bn, t.ms, obf, t.depth);
      return buf;
    }
    case FAM_DIRECT: {
      std::snprintf(buf, sizeof buf, "k_direct<%d, %d>", kDirectCfg[p.cfg].wk, p.pk > 1 ? 2 : obf);
      std::string r(buf);
      if (p.pk > 1) r += std::string(";k_reduce<") + b + ">";
      return r;
    }
    case FAM_DL: {
      const DlCfg& d = kDlCfg[p.cfg];
      std::snprintf(buf, sizeof buf, "%s<%d, %d, %d, %d, %d>", p.unal ? "k_dlu" : "k_dl", d.bm, d.bn, d.bk, d.stages,
                    p.pk > 1 ? 2 : obf);
      std::string r(buf);
      if (p.pk > 1) r += std::string(";k_reduce<") + b + ">";
      return r;
    }
    case FAM_DLSC: {
      const DlCfg& d = kDlCfg[p.cfg & 0xF];
      std::snprintf(buf, sizeof buf, "k_dl_sc<%d, %d, %d, %d>", d.bm, d.bn, d.bk, d.stages);
      return std::string(buf) + ";k_reduce<" + b + ">";
    }
    case FAM_TALL: {
      const TallCfg& t = kTallCfg[p.cfg];
      std::snprintf(buf, sizeof buf, "%s<%d, %d, %d, %d>", p.unal ? "k_tallu" : "k_tall", t.nt, t.bm, t.stages,
                    p.pk > 1 ? 2 : obf);
      std::string r(buf);
      if (p.pk > 1) r += std::string(";k_reduce<") + b + ">";
      return r;
    }
  }
  return "";
}

int config_index(int family, int cfg) {
  switch (family) {
    case FAM_TILE:
      return cfg >= 0 && cfg < N_TILE_CFG ? IDX_TILE + cfg : -1;
    case FAM_SKINNY_M:
      return cfg >= 0 && cfg < N_SKINNY_M_CFG ? IDX_SKINNY_M + cfg : -1;
    case FAM_SKINNY_N:
      return cfg >= 0 && cfg < N_SKINNY_N_CFG ? IDX_SKINNY_N + cfg : -1;
    case FAM_SMALLK:
      return cfg >= 0 && cfg < N_SMALLK_CFG ? IDX_SMALLK + cfg : -1;
    case FAM_STREAMK:
      return cfg >= 0 && cfg < N_STREAMK_CFG ? IDX_STREAMK + cfg : -1;
    case FAM_DIRECT:
      return cfg >= 0 && cfg < N_DIRECT_CFG ? IDX_DIRECT + cfg : -1;
    case FAM_PERSIST:
      return cfg >= 0 && cfg < N_TILE_CFG && kPersistCfg[cfg] ? IDX_PERSIST + cfg : -1;
    case FAM_DL:  // cfg | 0x100: the register-load form
      if ((cfg & 0x100) != 0) {
        const int c = cfg & 0xFF;
        return c < N_DL_CFG && kDlCfg[c].unal ? dlu_index(c) : -1;
      }
      return cfg >= 0 && cfg < N_DL_CFG ? IDX_DL + cfg : -1;
    case FAM_TALL:  // cfg | 0x100: the register-load form
      if ((cfg & 0x100) != 0) {
        const int c = cfg & 0xFF;
        return c < N_TALL_CFG && kTallCfg[c].unal ? tallu_index(c) : -1;
      }
      return cfg >= 0 && cfg < N_TALL_CFG ? IDX_TALL + cfg : -1;
    case FAM_DLSC:  // the direct-to-LDS configuration's costs (the same tile code)
      return ((cfg & 0xF) == 0 || (cfg & 0xF) == 4) && (cfg >> 4) <= 10 ? IDX_DL + (cfg & 0xF) : -1;
    case FAM_BATCHED:
    case FAM_GROUPED:  // the tile kernel's costs
      return cfg >= 0 && cfg < N_TILE_CFG && kGroupedCfg[cfg] ? IDX_TILE + cfg : -1;
  }
  return -1;
}

uint64_t shape_key(const Shape& s, bool* exact) {
  const int64_t lim = 1LL << 17;
  if (s.M < lim && s.N < lim && s.K < lim && s.dtype >= 0 && s.dtype < 16 && s.layouts < 4) {
    *exact = true;
    return (uint64_t)s.M | ((uint64_t)s.N << 17) | ((uint64_t)s.K << 34) | ((uint64_t)s.dtype << 51) |
           ((uint64_t)s.layouts << 55);
  }
  *exact = false;
  uint64_t h = 0x9E3779B97F4A7C15ull;
  const uint64_t v[5] = {(uint64_t)s.M, (uint64_t)s.N, (uint64_t)s.K, (uint64_t)s.dtype, (uint64_t)s.layouts};
  for (uint64_t x : v) {
    h ^= x + 0x9E3779B97F4A7C15ull + (h << 6) + (h >> 2);
    h *= 0xBF58476D1CE4E5B9ull;
  }
  return h | (1ull << 63);
}

// ---- paper arithmetic for explicit parameters ------------------------------

void taxonomy(const adaptcore_taxonomy_in_t& in, adaptcore_taxonomy_out_t* out) {
  out->pm = cdiv(in.M, in.m);
  out->pn = cdiv(in.N, in.n);
  out->pk = cdiv(in.K, in.k);
  out->acc_bytes = in.m1 * in.n1 * 4;
  const bool spatial = out->pm * out->pn >= in.n_core;
  const bool onchip = out->acc_bytes <= in.s_acc;
  out->cls = spatial ? (onchip ? AC_CLASS_COMMON : AC_CLASS_SINGLE_CORE_SPLITK)
                     : (onchip ? AC_CLASS_MULTI_CORE_SPLITK : AC_CLASS_HYBRID_SPLITK);
  // Eq. 1
  out->read_bytes = (double)in.elem_bytes * (double)in.M * (double)in.N * (double)in.K *
                    (1.0 / (double)in.m1 + 1.0 / (double)in.n1);
  const double MN = (double)in.M * (double)in.N;
  const double fin = (double)in.out_bytes * MN;
  switch (out->cls) {
    case AC_CLASS_COMMON:  // Eq. 2
      out->write_bytes = fin;
      break;
    case AC_CLASS_SINGLE_CORE_SPLITK:  // Eq. 3
      out->write_bytes = 4.0 * MN * (double)cdiv(in.K, in.k1) + fin;
      break;
    case AC_CLASS_MULTI_CORE_SPLITK:  // Eq. 4
      out->write_bytes = 4.0 * MN * (double)cdiv(in.K, in.k) + fin;
      break;
    default: {  // Eq. 5, each partition with its actual length
      double flushes = 0;
      for (int64_t p0 = 0; p0 < in.K; p0 += in.k) flushes += (double)cdiv(std::min(in.k, in.K - p0), in.k1);
      out->write_bytes = 4.0 * MN * flushes + fin;
    }
  }
}

double schedule(int kind, int64_t Q, int64_t L, double tm, double tp, double td) {
  switch (kind) {
    case 0:
      return (double)L * (tm + tp) + td;  // Eq. 12
    case 1:
      return tm + (double)(L - 1) * std::max(tm, tp) + tp + td;  // Eq. 13
    case 2:
      return tm + (double)(Q * L - 1) * std::max(tm, tp) + tp + (double)Q * td;  // Eq. 14
  }
  return -1.0;
}

}  // namespace ac
