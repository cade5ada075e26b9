// C ABI: validation, the plan cache (O(1) online dispatch of the online
// phase, Section 3.2), per-stream workspaces and the launch.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <atomic>
#include <chrono>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "adaptcore.h"
#include "noalloc.h"
#include "planner.h"
#include "registry.h"

struct adaptcore_plan_s {
  ac::Plan p;
};

namespace {

thread_local std::string t_err;
thread_local adaptcore_status t_status = AC_OK;
// adaptcore_set_override: VariantKey forced on this thread's adaptcore_plan
// calls (0 = none).
thread_local uint64_t t_override = 0;

void init_for_planning();

adaptcore_status fail(adaptcore_status st, const std::string& msg) {
  t_err = msg;
  t_status = st;
  return st;
}

std::mutex g_mu;  // planning, cache inserts, profile changes
adaptcore_hw_t g_hw = ac::default_hw();

std::atomic<uint64_t> st_lookups{0}, st_hits{0}, st_misses{0}, st_launches{0}, st_entries{0};
std::atomic<uint64_t> st_class[4];
double st_miss_seconds = 0;  // under g_mu

// ---- plan cache: open addressing, lock-free reads --------------------------
// A slot's key is published (release) after its plan pointer, so a reader that
// sees the key also sees the plan. The table only grows; replaced tables stay
// alive until adaptcore_cache_clear so concurrent readers never touch freed
// memory.
struct Slot {
  std::atomic<uint64_t> key{0};  // shape key + 1; 0 = empty
  std::atomic<adaptcore_plan_s*> plan{nullptr};
};
struct Table {
  size_t cap;
  size_t used = 0;
  Slot* slots;
  explicit Table(size_t c) : cap(c), slots(new Slot[c]) {}
  ~Table() { delete[] slots; }
};
std::atomic<Table*> g_tab{nullptr};
std::vector<Table*> g_retired;
std::vector<adaptcore_plan_s*> g_owned;
std::map<std::tuple<int64_t, int64_t, int64_t, int, uint32_t>, adaptcore_plan_s*> g_big;  // dims >= 2^17
std::map<std::pair<std::tuple<int64_t, int64_t, int64_t, int, uint32_t>, uint64_t>, adaptcore_plan_s*> g_forced;
// grouped plans: (rows, groups, N, K, dtype, layouts) [, forced key]
typedef std::tuple<int64_t, int64_t, int64_t, int64_t, int, uint32_t> GroupKey;
std::map<GroupKey, adaptcore_plan_s*> g_grouped;
std::map<std::pair<GroupKey, uint64_t>, adaptcore_plan_s*> g_grouped_forced;
std::map<GroupKey, adaptcore_plan_s*> g_batched;  // (M, batch, N, K, dtype, layouts)
std::map<std::pair<GroupKey, uint64_t>, adaptcore_plan_s*> g_batched_forced;

inline uint64_t mix(uint64_t x) {
  x ^= x >> 33;
  x *= 0xff51afd7ed558ccdull;
  x ^= x >> 33;
  x *= 0xc4ceb9fe1a85ec53ull;
  x ^= x >> 33;
  return x;
}

inline adaptcore_plan_s* table_find(const Table* t, uint64_t k) {
  if (!t) return nullptr;
  const size_t m = t->cap - 1;
  for (size_t i = mix(k) & m;; i = (i + 1) & m) {
    const uint64_t s = t->slots[i].key.load(std::memory_order_acquire);
    if (s == k) return t->slots[i].plan.load(std::memory_order_acquire);
    if (s == 0) return nullptr;
  }
}

void table_put(Table* t, uint64_t k, adaptcore_plan_s* p) {
  const size_t m = t->cap - 1;
  for (size_t i = mix(k) & m;; i = (i + 1) & m) {
    if (t->slots[i].key.load(std::memory_order_relaxed) == 0) {
      t->slots[i].plan.store(p, std::memory_order_relaxed);
      t->slots[i].key.store(k, std::memory_order_release);
      ++t->used;
      return;
    }
  }
}

// Under g_mu.
void cache_insert(uint64_t k, adaptcore_plan_s* p) {
  Table* t = g_tab.load(std::memory_order_relaxed);
  if (!t) {
    t = new Table(1024);
    g_tab.store(t, std::memory_order_release);
  }
  if ((t->used + 1) * 2 > t->cap) {
    Table* n = new Table(t->cap * 2);
    for (size_t i = 0; i < t->cap; ++i) {
      const uint64_t kk = t->slots[i].key.load(std::memory_order_relaxed);
      if (kk) table_put(n, kk, t->slots[i].plan.load(std::memory_order_relaxed));
    }
    g_tab.store(n, std::memory_order_release);
    g_retired.push_back(t);
    t = n;
  }
  table_put(t, k, p);
}

bool valid_args(int64_t M, int64_t N, int64_t K, int32_t dtype, uint32_t layouts, adaptcore_status* st) {
  const int64_t lim = (1LL << 31) - 1;
  if (M < 0 || N < 0 || K < 0 || M > lim || N > lim || K > lim) {
    *st = fail(AC_ERR_INVALID_VALUE, "dimensions must be in [0, 2^31)");
    return false;
  }
  if (dtype != AC_BF16_F32OUT && dtype != AC_BF16_BF16OUT && dtype != AC_F16_F32OUT && dtype != AC_F16_F16OUT) {
    *st = fail(AC_ERR_UNSUPPORTED, "dtype not provided by this build (bf16 or fp16 inputs, fp32 or 16-bit output)");
    return false;
  }
  if (layouts > AC_LAYOUT_COL_COL) {
    *st = fail(AC_ERR_UNSUPPORTED, "unknown layout bits");
    return false;
  }
  return true;
}

// Grouped and batched products read their operands row-major.
bool row_major_only(uint32_t layouts) {
  if (layouts == AC_LAYOUT_ROW_ROW) return true;
  fail(AC_ERR_UNSUPPORTED, "grouped and batched products take row-major A and B only");
  return false;
}

adaptcore_plan_s* plan_miss(const ac::Shape& s) {
  const auto t0 = std::chrono::steady_clock::now();
  int cls = 0;
  std::vector<ac::Plan> c = ac::enumerate(s, g_hw, &cls);
  if (c.empty()) return nullptr;
  auto* p = new adaptcore_plan_s{c.front()};
  bool exact;
  p->p.shape_key = ac::shape_key(s, &exact);
  g_owned.push_back(p);
  st_miss_seconds += std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
  st_misses.fetch_add(1, std::memory_order_relaxed);
  st_class[cls & 3].fetch_add(1, std::memory_order_relaxed);
  st_entries.fetch_add(1, std::memory_order_relaxed);
  return p;
}

inline const adaptcore_plan_s* lookup(int64_t M, int64_t N, int64_t K, int32_t dtype, uint32_t layouts) {
  st_lookups.fetch_add(1, std::memory_order_relaxed);
  const ac::Shape s{M, N, K, dtype, layouts};
  bool exact;
  const uint64_t key = ac::shape_key(s, &exact);
  if (exact) {
    if (adaptcore_plan_s* p = table_find(g_tab.load(std::memory_order_acquire), key + 1)) {
      st_hits.fetch_add(1, std::memory_order_relaxed);
      return p;
    }
  }
  init_for_planning();
  std::lock_guard<std::mutex> lk(g_mu);
  if (exact) {
    if (adaptcore_plan_s* p = table_find(g_tab.load(std::memory_order_acquire), key + 1)) {
      st_hits.fetch_add(1, std::memory_order_relaxed);
      return p;
    }
  } else {
    auto it = g_big.find(std::make_tuple(M, N, K, (int)dtype, layouts));
    if (it != g_big.end()) {
      st_hits.fetch_add(1, std::memory_order_relaxed);
      return it->second;
    }
  }
  adaptcore_plan_s* p = plan_miss(s);
  if (!p) {
    fail(AC_ERR_INTERNAL, "no legal configuration for the shape");
    return nullptr;
  }
  if (exact)
    cache_insert(key + 1, p);
  else
    g_big[std::make_tuple(M, N, K, (int)dtype, layouts)] = p;
  return p;
}

// ---- device and workspaces ------------------------------------------------
struct Workspace {
  char* ptr = nullptr;
  int64_t bytes = 0;
};
std::mutex g_ws_mu;
std::map<std::pair<int, void*>, Workspace> g_ws;
std::vector<char*> g_ws_retired;  // replaced workspaces, kept until the process ends
std::once_flag g_init_once;
adaptcore_status g_init_status = AC_ERR_NOT_INITIALIZED;
std::string g_init_msg;

adaptcore_status do_init() {
  int dev = 0, n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n <= 0) {
    g_init_msg = "no HIP device";
    return AC_ERR_NOT_INITIALIZED;
  }
  if (hipGetDevice(&dev) != hipSuccess) {
    g_init_msg = "hipGetDevice failed";
    return AC_ERR_NOT_INITIALIZED;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
    g_init_msg = "hipGetDeviceProperties failed";
    return AC_ERR_NOT_INITIALIZED;
  }
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) {
    g_init_msg = std::string("kernels are built for gfx950, device is ") + prop.gcnArchName;
    return AC_ERR_UNSUPPORTED;
  }
  ac::query_occupancy();
  // Resolve the no-allocation entry point's scratch array on this device
  // now; a failure is reported by that entry point (it tries again), the
  // rest of the library does not depend on it.
  void* scratch = nullptr;
  (void)ac::noalloc_scratch(dev, &scratch);
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_hw.n_cu != prop.multiProcessorCount) {
    g_hw.n_cu = prop.multiProcessorCount;
  }
  return AC_OK;
}

adaptcore_status ensure_init() {
  std::call_once(g_init_once, [] { g_init_status = do_init(); });
  if (g_init_status != AC_OK) return fail(g_init_status, g_init_msg);
  return AC_OK;
}

// Every planning path runs this first (outside g_mu), so a plan is priced
// with the occupancies the device reports for the compiled kernels whatever
// the order of the caller's first calls; host API queries only, no launch.
// Without a device the planner keeps its table of workgroups per CU.
void init_for_planning() { std::call_once(g_init_once, [] { g_init_status = do_init(); }); }

// Workspace of (current device, stream) with at least `need` bytes; allocates
// outside stream capture only. Partials are fully rewritten by every call that
// uses them, so a workspace needs no initialisation.
adaptcore_status get_workspace(hipStream_t stream, int64_t need, Workspace* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(AC_ERR_NOT_INITIALIZED, "hipGetDevice failed");
  std::lock_guard<std::mutex> lk(g_ws_mu);
  Workspace& w = g_ws[std::make_pair(dev, (void*)stream)];
  if (w.ptr && w.bytes >= need) {
    *out = w;
    return AC_OK;
  }
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cs) == hipSuccess && cs != hipStreamCaptureStatusNone)
    return fail(AC_ERR_NOT_INITIALIZED,
                "split-K workspace missing for this stream under capture: call adaptcore_reserve_workspace first");
  const int64_t grow = std::max<int64_t>(std::max<int64_t>(need, 1 << 20), w.bytes + w.bytes / 2);
  void* p = nullptr;
  if (hipMalloc(&p, (size_t)grow) != hipSuccess) return fail(AC_ERR_OUT_OF_MEMORY, "workspace allocation failed");
  // The replaced buffer is never freed: a graph captured earlier on this
  // stream, or another thread that took the pointer and has not launched
  // yet, may still use it. With growth by at least 1.5x the retired buffers
  // of a stream add up to at most twice its current workspace.
  if (w.ptr) g_ws_retired.push_back(w.ptr);
  w.ptr = static_cast<char*>(p);
  w.bytes = grow;
  *out = w;
  return AC_OK;
}

}  // namespace

extern "C" {

adaptcore_status adaptcore_init(void) { return ensure_init(); }

const adaptcore_plan_t* adaptcore_plan(int64_t M, int64_t N, int64_t K, int32_t dtype, uint32_t layouts) {
  adaptcore_status st;
  if (!valid_args(M, N, K, dtype, layouts, &st)) return nullptr;
  if (t_override != 0) return adaptcore_plan_variant(M, N, K, dtype, layouts, t_override);
  return lookup(M, N, K, dtype, layouts);
}

adaptcore_status adaptcore_set_override(uint64_t variant_key_or_0) {
  t_override = variant_key_or_0;
  return AC_OK;
}

uint64_t adaptcore_get_override(void) { return t_override; }

const adaptcore_plan_t* adaptcore_plan_variant(int64_t M, int64_t N, int64_t K, int32_t dtype, uint32_t layouts,
                                               uint64_t variant_key) {
  adaptcore_status st;
  if (!valid_args(M, N, K, dtype, layouts, &st)) return nullptr;
  const auto tk = std::make_tuple(M, N, K, (int)dtype, layouts);
  init_for_planning();
  std::lock_guard<std::mutex> lk(g_mu);
  auto it = g_forced.find(std::make_pair(tk, variant_key));
  if (it != g_forced.end()) return it->second;
  ac::Plan p;
  const ac::Shape s{M, N, K, dtype, layouts};
  if (!ac::plan_for_key(s, g_hw, variant_key, &p)) {
    fail(AC_ERR_INVALID_VALUE, "variant key is not legal for this shape");
    return nullptr;
  }
  bool exact;
  p.shape_key = ac::shape_key(s, &exact);
  auto* pp = new adaptcore_plan_s{p};
  g_owned.push_back(pp);
  g_forced[std::make_pair(tk, variant_key)] = pp;
  return pp;
}

adaptcore_status adaptcore_reserve_workspace(void* stream, int64_t bytes) {
  if (bytes < 0) return fail(AC_ERR_INVALID_VALUE, "negative workspace size");
  adaptcore_status st = ensure_init();
  if (st != AC_OK) return st;
  Workspace w;
  return get_workspace(static_cast<hipStream_t>(stream), bytes, &w);
}

}  // extern "C"

namespace {

// One call of a plain plan; epi != 0 selects the AddMM epilogue. With
// `fixed` the workspace is the device scratch array of
// adaptcore_matmul_noalloc (nothing is allocated).
adaptcore_status run_matmul(const adaptcore_plan_t* plan, const void* A, int64_t lda, const void* B, int64_t ldb,
                            void* C, int64_t ldc, void* stream, int epi, float alpha, float beta, const float* bias,
                            bool fixed = false) {
  if (!plan) return fail(AC_ERR_INVALID_VALUE, "null plan");
  const ac::Plan& p = plan->p;
  if (p.family == ac::FAM_GROUPED)
    return fail(AC_ERR_INVALID_VALUE, "grouped plan: run it with adaptcore_grouped_matmul");
  if (p.family == ac::FAM_BATCHED)
    return fail(AC_ERR_INVALID_VALUE, "batched plan: run it with adaptcore_batched_matmul");
  const int64_t M = p.s.M, N = p.s.N, K = p.s.K;
  if (M == 0 || N == 0) return AC_OK;
  const bool a_col = (p.s.layouts & AC_LAYOUT_A_COL) != 0, b_col = (p.s.layouts & AC_LAYOUT_B_COL) != 0;
  if (lda < std::max<int64_t>(1, a_col ? M : K) || ldb < std::max<int64_t>(1, b_col ? K : N) ||
      ldc < std::max<int64_t>(1, N))
    return fail(AC_ERR_INVALID_VALUE, "leading dimension smaller than the stored row or column");
  // the kernels address A and B tiles with 32-bit byte offsets from a row
  // base (of the caller's operand, or of the row-major copy of a column-major
  // one, whose rows are padded to a multiple of 8)
  if ((a_col ? (K + 7) / 8 * 8 : lda) >= AC_MAX_LD || (b_col ? (N + 7) / 8 * 8 : ldb) >= AC_MAX_LD)
    return fail(AC_ERR_UNSUPPORTED, "row pitch of A or B must be below 2^23 elements");
  if (!C || (K > 0 && (!A || !B))) return fail(AC_ERR_INVALID_VALUE, "null matrix pointer");
  const int cbytes = ac::dtype_out_bytes(p.s.dtype);
  if (((uintptr_t)A & 1) || ((uintptr_t)B & 1) || ((uintptr_t)C & (cbytes - 1)))
    return fail(AC_ERR_INVALID_VALUE, "pointer not aligned to its element size");
  adaptcore_status st = ensure_init();
  if (st != AC_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);

  ac::GemmArgs g;
  std::memset(&g, 0, sizeof g);
  g.A = static_cast<const uint16_t*>(A);
  g.B = static_cast<const uint16_t*>(B);
  g.C = C;
  g.M = M;
  g.N = N;
  g.K = K;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = ldc;
  g.ldw = (N + 7) / 8 * 8;
  g.epi = epi;
  g.alpha = alpha;
  g.beta = beta;
  g.bias = bias;
  g.kB = K;
  g.nB = N;
  // Direct-to-LDS plans: operands the plan does not copy must have 16-byte
  // aligned rows of whole chunks; otherwise the configuration's register-load
  // form (if it has one, and the operands are row-major with K, N >= 8), else
  // the register-staged sibling of the same tiling, runs on the operands as
  // given (no padding copies).
  // Off-chip accumulation plans load like the direct-to-LDS ones; with such
  // operands the direct-to-LDS split-K plan of the same slices (same
  // partials, same sum) runs instead, with its own fallbacks below.
  ac::Plan sib, dl_base;
  const ac::Plan* src = &p;
  if (p.family == ac::FAM_DLSC) {
    const bool a_ok = a_col || p.ws_a_off >= 0 || ac::dl_a_aligned(A, lda, K);
    const bool b_ok = b_col || p.ws_b_off >= 0 || ac::dl_b_aligned(B, ldb, N);
    if (!(a_ok && b_ok)) {
      adaptcore_hw_t hw;
      {
        std::lock_guard<std::mutex> lk(g_mu);
        hw = g_hw;
      }
      const uint64_t key = ac::make_variant_key(ac::FAM_DL, p.cfg & 0xF, 0, p.pk, p.s.dtype, (int)p.s.layouts);
      if (!ac::plan_for_key(p.s, hw, key, &dl_base))
        return fail(AC_ERR_UNSUPPORTED, "operands not aligned for this plan and no fallback applies");
      src = &dl_base;
    }
  }
  const ac::Plan* run = src;
  bool dl = src->family == ac::FAM_DL || src->family == ac::FAM_DLSC;
  if (src->family == ac::FAM_DL && !src->unal) {  // (the register-load form takes any alignment)
    const bool a_ok = a_col || src->ws_a_off >= 0 || ac::dl_a_aligned(A, lda, K);
    const bool b_ok = b_col || src->ws_b_off >= 0 || ac::dl_b_aligned(B, ldb, N);
    if (!(a_ok && b_ok)) {
      sib = *src;
      const ac::DlCfg& d = ac::kDlCfg[src->cfg];
      // (column-major operands reach the kernel as aligned row-major copies)
      if (d.unal && K >= 8 && N >= 8) {
        sib.unal = 1;
      } else if (d.sibling >= 0) {
        sib.family = ac::FAM_TILE;
        sib.cfg = d.sibling;
        dl = false;
      } else {
        return fail(AC_ERR_UNSUPPORTED, "operands not aligned for this configuration and no fallback applies");
      }
      run = &sib;
    }
  }
  // Tall-skinny plans of the direct-load form need A with 16-byte aligned
  // rows; otherwise the configuration's register-load form runs if it has
  // one, else the skinny-N kernel (any alignment) with the same split count
  // if it has one, else unsplit.
  if (p.family == ac::FAM_TALL && !p.unal && !ac::tall_a_aligned(A, lda, K) && ac::kTallCfg[p.cfg].unal) {
    sib = p;
    sib.unal = 1;
    run = &sib;
  } else if (p.family == ac::FAM_TALL && !p.unal && !ac::tall_a_aligned(A, lda, K)) {
    adaptcore_hw_t hw;
    {
      std::lock_guard<std::mutex> lk(g_mu);
      hw = g_hw;
    }
    const int cfg = ac::kTallCfg[p.cfg].nt - 1;  // skinny-N configuration of the same column count
    bool ok = false;
    for (int pk : {p.pk, 1}) {
      const uint64_t key = ac::make_variant_key(ac::FAM_SKINNY_N, cfg, 0, pk, p.s.dtype, (int)p.s.layouts);
      if ((ok = ac::plan_for_key(p.s, hw, key, &sib))) break;
    }
    if (!ok) return fail(AC_ERR_UNSUPPORTED, "A not aligned for this plan and no fallback applies");
    run = &sib;
  }
  // the launch fields, workspace and prologue of the plan that runs
  const ac::Plan& q = *run;
  g.pk = q.family == ac::FAM_STREAMK ? 1 : q.pk;
  g.kper = q.kper;
  g.tiles_m = q.pm;
  g.tiles_n = q.pn;
  g.swizzle = q.swizzle;
  g.iters_per_wg = q.iters_per_wg;
  g.sk_tiles = q.sk_tiles;
  g.ws_pk = q.ws_pk;
  g.grid = q.grid_x;
  if (q.ws_bytes > 0) {
    Workspace w;
    if (fixed) {
      if (q.ws_bytes > ac::NOALLOC_SCRATCH_BYTES)
        return fail(AC_ERR_UNSUPPORTED, "the plan's workspace (" + std::to_string(q.ws_bytes) +
                                            " bytes) exceeds the no-allocation scratch of " +
                                            std::to_string(ac::NOALLOC_SCRATCH_BYTES) + " bytes");
      int dev = 0;
      void* ptr = nullptr;
      if (hipGetDevice(&dev) != hipSuccess || ac::noalloc_scratch(dev, &ptr) != hipSuccess)
        return fail(AC_ERR_NOT_INITIALIZED, "the device scratch array is not addressable on this device");
      w.ptr = static_cast<char*>(ptr);
      w.bytes = ac::NOALLOC_SCRATCH_BYTES;
    } else {
      st = get_workspace(s, q.ws_bytes, &w);
      if (st != AC_OK) return st;
    }
    g.ws = reinterpret_cast<float*>(w.ptr);
    char* base = static_cast<char*>(w.ptr);
    // prologue: row-major copies of column-major operands, and zero-padded
    // copies of unaligned row-major operands for the direct loads of a
    // direct-to-LDS plan (rows of K and N rounded up to 8); the register-load
    // form and the sibling read the row-major operands as given. A
    // tall-skinny plan reads B's transposed copy (N x K8).
    const bool pads = dl && !run->unal;
    const bool tall = q.family == ac::FAM_TALL;
    const int64_t K8 = (K + 7) / 8 * 8, N8 = (N + 7) / 8 * 8;
    if (tall && q.ws_b_off >= 0) {
      uint16_t* bt = reinterpret_cast<uint16_t*>(base + q.ws_b_off);
      const hipError_t e = b_col ? ac::launch_pad16(g.B, ldb, N, K, bt, K8, s)
                                 : ac::launch_transpose16(g.B, ldb, K, N, bt, K8, s);
      if (e != hipSuccess) return fail(AC_ERR_LAUNCH, std::string("kernel launch failed: ") + hipGetErrorString(e));
      g.B = bt;
      g.ldb = K8;
    }
    if (q.ws_a_off >= 0 && (a_col || pads)) {
      uint16_t* a2 = reinterpret_cast<uint16_t*>(base + q.ws_a_off);
      const hipError_t e = a_col ? ac::launch_transpose16(g.A, lda, K, M, a2, K8, s)
                                 : ac::launch_pad16(g.A, lda, M, K, a2, K8, s);
      if (e != hipSuccess) return fail(AC_ERR_LAUNCH, std::string("kernel launch failed: ") + hipGetErrorString(e));
      g.A = a2;
      g.lda = K8;
    }
    if (!tall && q.ws_b_off >= 0 && (b_col || pads)) {
      uint16_t* b2 = reinterpret_cast<uint16_t*>(base + q.ws_b_off);
      const hipError_t e = b_col ? ac::launch_transpose16(g.B, ldb, N, K, b2, N8, s)
                                 : ac::launch_pad16(g.B, ldb, K, N, b2, N8, s);
      if (e != hipSuccess) return fail(AC_ERR_LAUNCH, std::string("kernel launch failed: ") + hipGetErrorString(e));
      g.B = b2;
      g.ldb = N8;
      if (pads) g.nB = N8;
    }
    // the direct loads run over whole 8-element chunks of A's rows (zeros
    // past K in a copy); B's rows stay K. The register-load form reads the
    // operands as given and zero-fills past K itself.
    if (pads) g.K = K8;
  }
  const hipError_t e =
      ac::dtype_f16_input(p.s.dtype) ? ac::f16::launch_plan(*run, g, s) : ac::launch_plan(*run, g, s);
  if (e != hipSuccess) return fail(AC_ERR_LAUNCH, std::string("kernel launch failed: ") + hipGetErrorString(e));
  st_launches.fetch_add((uint64_t)q.n_launch, std::memory_order_relaxed);
  return AC_OK;
}

}  // namespace

extern "C" {

adaptcore_status adaptcore_matmul(const adaptcore_plan_t* plan, const void* A, int64_t lda, const void* B, int64_t ldb,
                                  void* C, int64_t ldc, void* stream) {
  return run_matmul(plan, A, lda, B, ldb, C, ldc, stream, 0, 1.0f, 0.0f, nullptr);
}

adaptcore_status adaptcore_matmul_noalloc(const adaptcore_plan_t* plan, const void* A, int64_t lda, const void* B,
                                          int64_t ldb, void* C, int64_t ldc, void* stream) {
  return run_matmul(plan, A, lda, B, ldb, C, ldc, stream, 0, 1.0f, 0.0f, nullptr, true);
}

int64_t adaptcore_noalloc_scratch_bytes(void) { return ac::NOALLOC_SCRATCH_BYTES; }

adaptcore_status adaptcore_addmm(const adaptcore_plan_t* plan, const void* A, int64_t lda, const void* B, int64_t ldb,
                                 void* C, int64_t ldc, float alpha, float beta, const float* bias, void* stream) {
  if (!std::isfinite(alpha) || !std::isfinite(beta)) return fail(AC_ERR_INVALID_VALUE, "alpha and beta must be finite");
  if (((uintptr_t)bias & 3)) return fail(AC_ERR_INVALID_VALUE, "bias not aligned to 4 bytes");
  return run_matmul(plan, A, lda, B, ldb, C, ldc, stream, 1, alpha, beta, bias);
}

const adaptcore_plan_t* adaptcore_grouped_plan(int64_t rows, int64_t groups, int64_t N, int64_t K, int32_t dtype,
                                               uint32_t layouts) {
  adaptcore_status st;
  if (!valid_args(rows, N, K, dtype, layouts, &st)) return nullptr;
  if (!row_major_only(layouts)) return nullptr;
  if (groups < 0 || groups > (1LL << 20)) {
    fail(AC_ERR_INVALID_VALUE, "groups must be in [0, 2^20]");
    return nullptr;
  }
  st_lookups.fetch_add(1, std::memory_order_relaxed);
  const GroupKey k = std::make_tuple(rows, groups, N, K, (int)dtype, layouts);
  init_for_planning();
  std::lock_guard<std::mutex> lk(g_mu);
  auto it = g_grouped.find(k);
  if (it != g_grouped.end()) {
    st_hits.fetch_add(1, std::memory_order_relaxed);
    return it->second;
  }
  const auto t0 = std::chrono::steady_clock::now();
  ac::Plan p;
  const ac::Shape s{rows, N, K, dtype, layouts};
  if (!ac::plan_grouped(s, groups, g_hw, &p)) {
    fail(AC_ERR_UNSUPPORTED, "no grouped configuration fits (launch grid too large)");
    return nullptr;
  }
  bool exact;
  p.shape_key = ac::shape_key(s, &exact);
  auto* pp = new adaptcore_plan_s{p};
  g_owned.push_back(pp);
  g_grouped[k] = pp;
  st_miss_seconds += std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
  st_misses.fetch_add(1, std::memory_order_relaxed);
  st_entries.fetch_add(1, std::memory_order_relaxed);
  return pp;
}

const adaptcore_plan_t* adaptcore_grouped_plan_variant(int64_t rows, int64_t groups, int64_t N, int64_t K,
                                                       int32_t dtype, uint32_t layouts, uint64_t variant_key) {
  adaptcore_status st;
  if (!valid_args(rows, N, K, dtype, layouts, &st)) return nullptr;
  if (!row_major_only(layouts)) return nullptr;
  if (groups < 0 || groups > (1LL << 20)) {
    fail(AC_ERR_INVALID_VALUE, "groups must be in [0, 2^20]");
    return nullptr;
  }
  const GroupKey k = std::make_tuple(rows, groups, N, K, (int)dtype, layouts);
  init_for_planning();
  std::lock_guard<std::mutex> lk(g_mu);
  auto it = g_grouped_forced.find(std::make_pair(k, variant_key));
  if (it != g_grouped_forced.end()) return it->second;
  ac::Plan p;
  const ac::Shape s{rows, N, K, dtype, layouts};
  if (!ac::grouped_for_key(s, groups, g_hw, variant_key, &p)) {
    fail(AC_ERR_INVALID_VALUE, "variant key is not a legal grouped configuration");
    return nullptr;
  }
  bool exact;
  p.shape_key = ac::shape_key(s, &exact);
  auto* pp = new adaptcore_plan_s{p};
  g_owned.push_back(pp);
  g_grouped_forced[std::make_pair(k, variant_key)] = pp;
  return pp;
}

}  // extern "C"

namespace {

// One call of a grouped plan; epi != 0 selects the AddMM epilogue (bias rows
// stride_bias apart, one per group).
adaptcore_status run_grouped(const adaptcore_plan_t* plan, const int32_t* counts, const void* A, int64_t lda,
                             const void* B, int64_t ldb, int64_t stride_b, void* C, int64_t ldc, void* stream,
                             int epi, float alpha, float beta, const float* bias, int64_t stride_bias) {
  if (!plan) return fail(AC_ERR_INVALID_VALUE, "null plan");
  const ac::Plan& p = plan->p;
  if (p.family != ac::FAM_GROUPED)
    return fail(AC_ERR_INVALID_VALUE, "not a grouped plan: run it with adaptcore_matmul");
  const int64_t rows = p.s.M, N = p.s.N, K = p.s.K;
  if (lda < std::max<int64_t>(1, K) || ldb < std::max<int64_t>(1, N) || ldc < std::max<int64_t>(1, N))
    return fail(AC_ERR_INVALID_VALUE, "leading dimension smaller than the row length");
  if (stride_b < 0 || stride_b >= (1LL << 40)) return fail(AC_ERR_INVALID_VALUE, "stride_b must be in [0, 2^40)");
  if (lda >= AC_MAX_LD || ldb >= AC_MAX_LD)
    return fail(AC_ERR_UNSUPPORTED, "lda and ldb must be below 2^23 elements");
  if (rows == 0 || p.groups == 0 || N == 0 || p.grid_x == 0) return AC_OK;
  if (!C || !counts || (K > 0 && (!A || !B))) return fail(AC_ERR_INVALID_VALUE, "null pointer");
  const int cbytes = ac::dtype_out_bytes(p.s.dtype);
  if (((uintptr_t)A & 1) || ((uintptr_t)B & 1) || ((uintptr_t)C & (cbytes - 1)) || ((uintptr_t)counts & 3))
    return fail(AC_ERR_INVALID_VALUE, "pointer not aligned to its element size");
  adaptcore_status st = ensure_init();
  if (st != AC_OK) return st;

  ac::GroupArgs a;
  std::memset(&a, 0, sizeof a);
  a.g.A = static_cast<const uint16_t*>(A);
  a.g.B = static_cast<const uint16_t*>(B);
  a.g.C = C;
  a.g.M = rows;
  a.g.N = N;
  a.g.K = K;
  a.g.lda = lda;
  a.g.ldb = ldb;
  a.g.ldc = ldc;
  a.g.pk = 1;
  a.g.kper = p.kper;
  a.g.tiles_m = p.pm;
  a.g.tiles_n = p.pn;
  a.g.swizzle = p.swizzle;
  a.g.epi = epi;
  a.g.alpha = alpha;
  a.g.beta = beta;
  a.g.bias = bias;
  a.counts = counts;
  a.rows = rows;
  a.stride_b = stride_b;
  a.stride_bias = stride_bias;
  a.groups = (int)p.groups;
  a.slots = p.pm;
  const hipError_t e = ac::dtype_f16_input(p.s.dtype) ? ac::f16::launch_grouped_plan(p, a, static_cast<hipStream_t>(stream))
                                                       : ac::launch_grouped_plan(p, a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(AC_ERR_LAUNCH, std::string("kernel launch failed: ") + hipGetErrorString(e));
  st_launches.fetch_add(1, std::memory_order_relaxed);
  return AC_OK;
}

}  // namespace

extern "C" {

adaptcore_status adaptcore_grouped_matmul(const adaptcore_plan_t* plan, const int32_t* counts, const void* A,
                                          int64_t lda, const void* B, int64_t ldb, int64_t stride_b, void* C,
                                          int64_t ldc, void* stream) {
  return run_grouped(plan, counts, A, lda, B, ldb, stride_b, C, ldc, stream, 0, 1.0f, 0.0f, nullptr, 0);
}

adaptcore_status adaptcore_grouped_addmm(const adaptcore_plan_t* plan, const int32_t* counts, const void* A,
                                         int64_t lda, const void* B, int64_t ldb, int64_t stride_b, void* C,
                                         int64_t ldc, float alpha, float beta, const float* bias, int64_t stride_bias,
                                         void* stream) {
  if (!std::isfinite(alpha) || !std::isfinite(beta)) return fail(AC_ERR_INVALID_VALUE, "alpha and beta must be finite");
  if (((uintptr_t)bias & 3)) return fail(AC_ERR_INVALID_VALUE, "bias not aligned to 4 bytes");
  if (stride_bias < 0 || stride_bias >= (1LL << 40))
    return fail(AC_ERR_INVALID_VALUE, "stride_bias must be in [0, 2^40)");
  return run_grouped(plan, counts, A, lda, B, ldb, stride_b, C, ldc, stream, 1, alpha, beta, bias, stride_bias);
}

const adaptcore_plan_t* adaptcore_batched_plan(int64_t batch, int64_t M, int64_t N, int64_t K, int32_t dtype,
                                               uint32_t layouts) {
  adaptcore_status st;
  if (!valid_args(M, N, K, dtype, layouts, &st)) return nullptr;
  if (!row_major_only(layouts)) return nullptr;
  if (batch < 0 || batch > (1LL << 24)) {
    fail(AC_ERR_INVALID_VALUE, "batch must be in [0, 2^24]");
    return nullptr;
  }
  st_lookups.fetch_add(1, std::memory_order_relaxed);
  const GroupKey k = std::make_tuple(M, batch, N, K, (int)dtype, layouts);
  init_for_planning();
  std::lock_guard<std::mutex> lk(g_mu);
  auto it = g_batched.find(k);
  if (it != g_batched.end()) {
    st_hits.fetch_add(1, std::memory_order_relaxed);
    return it->second;
  }
  const auto t0 = std::chrono::steady_clock::now();
  ac::Plan p;
  const ac::Shape s{M, N, K, dtype, layouts};
  if (!ac::plan_batched(s, batch, g_hw, &p)) {
    fail(AC_ERR_UNSUPPORTED, "no batched configuration fits (launch grid too large)");
    return nullptr;
  }
  bool exact;
  p.shape_key = ac::shape_key(s, &exact);
  auto* pp = new adaptcore_plan_s{p};
  g_owned.push_back(pp);
  g_batched[k] = pp;
  st_miss_seconds += std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
  st_misses.fetch_add(1, std::memory_order_relaxed);
  st_entries.fetch_add(1, std::memory_order_relaxed);
  return pp;
}

const adaptcore_plan_t* adaptcore_batched_plan_variant(int64_t batch, int64_t M, int64_t N, int64_t K,
                                                       int32_t dtype, uint32_t layouts, uint64_t variant_key) {
  adaptcore_status st;
  if (!valid_args(M, N, K, dtype, layouts, &st)) return nullptr;
  if (!row_major_only(layouts)) return nullptr;
  if (batch < 0 || batch > (1LL << 24)) {
    fail(AC_ERR_INVALID_VALUE, "batch must be in [0, 2^24]");
    return nullptr;
  }
  const GroupKey k = std::make_tuple(M, batch, N, K, (int)dtype, layouts);
  init_for_planning();
  std::lock_guard<std::mutex> lk(g_mu);
  auto it = g_batched_forced.find(std::make_pair(k, variant_key));
  if (it != g_batched_forced.end()) return it->second;
  ac::Plan p;
  const ac::Shape s{M, N, K, dtype, layouts};
  if (!ac::batched_for_key(s, batch, g_hw, variant_key, &p)) {
    fail(AC_ERR_INVALID_VALUE, "variant key is not a legal batched configuration");
    return nullptr;
  }
  bool exact;
  p.shape_key = ac::shape_key(s, &exact);
  auto* pp = new adaptcore_plan_s{p};
  g_owned.push_back(pp);
  g_batched_forced[std::make_pair(k, variant_key)] = pp;
  return pp;
}

}  // extern "C"

namespace {

// One call of a batched plan; epi != 0 selects the AddMM epilogue.
adaptcore_status run_batched(const adaptcore_plan_t* plan, const void* A, int64_t lda, int64_t stride_a,
                             const void* B, int64_t ldb, int64_t stride_b, void* C, int64_t ldc, int64_t stride_c,
                             void* stream, int epi, float alpha, float beta, const float* bias) {
  if (!plan) return fail(AC_ERR_INVALID_VALUE, "null plan");
  const ac::Plan& p = plan->p;
  if (p.family != ac::FAM_BATCHED)
    return fail(AC_ERR_INVALID_VALUE, "not a batched plan (adaptcore_batched_plan)");
  const int64_t M = p.s.M, N = p.s.N, K = p.s.K, batch = p.groups;
  if (lda < std::max<int64_t>(1, K) || ldb < std::max<int64_t>(1, N) || ldc < std::max<int64_t>(1, N))
    return fail(AC_ERR_INVALID_VALUE, "leading dimension smaller than the row length");
  const int64_t lim = 1LL << 40;
  if (stride_a < 0 || stride_b < 0 || stride_c < 0 || stride_a >= lim || stride_b >= lim || stride_c >= lim)
    return fail(AC_ERR_INVALID_VALUE, "batch strides must be in [0, 2^40)");
  if (batch > 1 && M > 0 && N > 0 && stride_c < (M - 1) * ldc + N)
    return fail(AC_ERR_INVALID_VALUE, "the C matrices of two batches overlap (stride_c too small)");
  if (lda >= AC_MAX_LD || ldb >= AC_MAX_LD)
    return fail(AC_ERR_UNSUPPORTED, "lda and ldb must be below 2^23 elements");
  if (batch == 0 || M == 0 || N == 0 || p.grid_x == 0) return AC_OK;
  if (!C || (K > 0 && (!A || !B))) return fail(AC_ERR_INVALID_VALUE, "null matrix pointer");
  const int cbytes = ac::dtype_out_bytes(p.s.dtype);
  if (((uintptr_t)A & 1) || ((uintptr_t)B & 1) || ((uintptr_t)C & (cbytes - 1)))
    return fail(AC_ERR_INVALID_VALUE, "pointer not aligned to its element size");
  adaptcore_status st = ensure_init();
  if (st != AC_OK) return st;

  ac::GroupArgs a;
  std::memset(&a, 0, sizeof a);
  a.g.A = static_cast<const uint16_t*>(A);
  a.g.B = static_cast<const uint16_t*>(B);
  a.g.C = C;
  a.g.M = M;
  a.g.N = N;
  a.g.K = K;
  a.g.lda = lda;
  a.g.ldb = ldb;
  a.g.ldc = ldc;
  a.g.pk = 1;
  a.g.kper = p.kper;
  a.g.tiles_m = p.pm;
  a.g.tiles_n = p.pn;
  a.g.swizzle = p.swizzle;
  a.g.epi = epi;
  a.g.alpha = alpha;
  a.g.beta = beta;
  a.g.bias = bias;
  a.counts = nullptr;
  a.rows = M;
  a.stride_a = stride_a;
  a.stride_b = stride_b;
  a.stride_c = stride_c;
  a.groups = (int)batch;
  a.slots = p.pm;
  a.tiles_per_group = (int)((M + p.tile_m - 1) / p.tile_m);
  const hipError_t e = ac::dtype_f16_input(p.s.dtype) ? ac::f16::launch_grouped_plan(p, a, static_cast<hipStream_t>(stream))
                                                       : ac::launch_grouped_plan(p, a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(AC_ERR_LAUNCH, std::string("kernel launch failed: ") + hipGetErrorString(e));
  st_launches.fetch_add(1, std::memory_order_relaxed);
  return AC_OK;
}

}  // namespace

extern "C" {

adaptcore_status adaptcore_batched_matmul(const adaptcore_plan_t* plan, const void* A, int64_t lda, int64_t stride_a,
                                          const void* B, int64_t ldb, int64_t stride_b, void* C, int64_t ldc,
                                          int64_t stride_c, void* stream) {
  return run_batched(plan, A, lda, stride_a, B, ldb, stride_b, C, ldc, stride_c, stream, 0, 1.0f, 0.0f, nullptr);
}

adaptcore_status adaptcore_batched_addmm(const adaptcore_plan_t* plan, const void* A, int64_t lda, int64_t stride_a,
                                         const void* B, int64_t ldb, int64_t stride_b, void* C, int64_t ldc,
                                         int64_t stride_c, float alpha, float beta, const float* bias, void* stream) {
  if (!std::isfinite(alpha) || !std::isfinite(beta)) return fail(AC_ERR_INVALID_VALUE, "alpha and beta must be finite");
  if (((uintptr_t)bias & 3)) return fail(AC_ERR_INVALID_VALUE, "bias not aligned to 4 bytes");
  return run_batched(plan, A, lda, stride_a, B, ldb, stride_b, C, ldc, stride_c, stream, 1, alpha, beta, bias);
}

adaptcore_status adaptcore_plan_info(const adaptcore_plan_t* plan, adaptcore_plan_desc_t* out) {
  if (!plan || !out) return fail(AC_ERR_INVALID_VALUE, "null argument");
  const ac::Plan& p = plan->p;
  std::memset(out, 0, sizeof *out);
  out->M = p.s.M;
  out->N = p.s.N;
  out->K = p.s.K;
  out->dtype = p.s.dtype;
  out->layouts = p.s.layouts;
  out->shape_key = p.shape_key;
  out->variant_key = p.variant_key;
  out->cls = p.cls;
  out->family = p.family;
  out->tile_m = p.tile_m;
  out->tile_n = p.tile_n;
  out->tile_k = p.tile_k;
  out->pm = p.pm;
  out->pn = p.pn;
  out->pk = p.family == ac::FAM_STREAMK ? p.ws_pk : p.pk;
  out->grid_x = p.grid_x;
  out->grid_y = p.grid_y;
  out->swizzle = p.swizzle;
  out->n_candidates = p.n_candidates;
  out->predicted_s = p.predicted;
  out->workspace_bytes = p.ws_bytes;
  out->groups = p.groups;
  return AC_OK;
}

adaptcore_status adaptcore_plan_kernels(const adaptcore_plan_t* plan, char* buf, int64_t len) {
  if (!plan || !buf) return fail(AC_ERR_INVALID_VALUE, "null argument");
  const std::string names = ac::kernel_names(plan->p);
  if (len < (int64_t)names.size() + 1) return fail(AC_ERR_INVALID_VALUE, "buffer too small");
  std::memcpy(buf, names.c_str(), names.size() + 1);
  return AC_OK;
}

int64_t adaptcore_candidates(int64_t M, int64_t N, int64_t K, int32_t dtype, uint32_t layouts,
                             adaptcore_candidate_t* out, int64_t cap) {
  adaptcore_status st;
  if (!valid_args(M, N, K, dtype, layouts, &st)) return st;
  adaptcore_hw_t hw;
  init_for_planning();
  {
    std::lock_guard<std::mutex> lk(g_mu);
    hw = g_hw;
  }
  const ac::Shape s{M, N, K, dtype, layouts};
  std::vector<ac::Plan> c = ac::enumerate(s, hw, nullptr);
  for (int64_t i = 0; i < (int64_t)c.size() && i < cap && out; ++i) {
    const ac::Plan& p = c[i];
    adaptcore_candidate_t& o = out[i];
    o.variant_key = p.variant_key;
    o.cls = p.cls;
    o.family = p.family;
    o.tile_m = p.tile_m;
    o.tile_n = p.tile_n;
    o.tile_k = p.tile_k;
    o.pk = p.family == ac::FAM_STREAMK ? p.ws_pk : p.pk;
    o.grid_x = p.grid_x;
    o.grid_y = p.grid_y;
    o.predicted_s = p.predicted;
  }
  return (int64_t)c.size();
}

adaptcore_status adaptcore_get_hw(adaptcore_hw_t* out) {
  if (!out) return fail(AC_ERR_INVALID_VALUE, "null argument");
  std::lock_guard<std::mutex> lk(g_mu);
  *out = g_hw;
  return AC_OK;
}

adaptcore_status adaptcore_set_hw(const adaptcore_hw_t* hw) {
  if (!hw) return fail(AC_ERR_INVALID_VALUE, "null argument");
  if (hw->n_cu <= 0 || hw->lds_bytes <= 0 || hw->s_acc_bytes <= 0 || !(hw->clock_hz > 0) || !(hw->hbm_bw > 0) ||
      !(hw->hbm_eta > 0) || !(hw->l2_bw_cu > 0) || !(hw->mfma_eta > 0) || !(hw->lds_bw_cu > 0) ||
      !(hw->unaligned_eta > 0) || hw->l2_hit < 0 || hw->l2_hit > 1 || hw->t_launch < 0 || hw->t_mem_latency < 0 ||
      hw->t_wg < 0 || !(hw->swizzle_gain > 0 && hw->swizzle_gain <= 1))
    return fail(AC_ERR_INVALID_VALUE, "profile field out of range");
  for (int i = 0; i < AC_N_CFG; ++i)
    if (!(hw->cfg_iter[i] >= 0 && hw->cfg_iter[i] < 1) || !(hw->cfg_wg[i] >= 0 && hw->cfg_wg[i] < 1) ||
        !(hw->cfg_wr[i] >= 0 && hw->cfg_wr[i] <= 1))
      return fail(AC_ERR_INVALID_VALUE, "calibrated configuration cost out of range");
  init_for_planning();  // the device's CU count must not replace the caller's profile later
  adaptcore_cache_clear();
  std::lock_guard<std::mutex> lk(g_mu);
  g_hw = *hw;
  return AC_OK;
}

adaptcore_status adaptcore_stats(adaptcore_stats_t* out) {
  if (!out) return fail(AC_ERR_INVALID_VALUE, "null argument");
  std::memset(out, 0, sizeof *out);
  out->lookups = st_lookups.load();
  out->hits = st_hits.load();
  out->misses = st_misses.load();
  out->entries = st_entries.load();
  out->launches = st_launches.load();
  for (int i = 0; i < 4; ++i) out->class_count[i] = st_class[i].load();
  std::lock_guard<std::mutex> lk(g_mu);
  out->miss_seconds = st_miss_seconds;
  return AC_OK;
}

adaptcore_status adaptcore_cache_clear(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  Table* t = g_tab.exchange(nullptr);
  delete t;
  for (Table* r : g_retired) delete r;
  g_retired.clear();
  for (adaptcore_plan_s* p : g_owned) delete p;
  g_owned.clear();
  g_big.clear();
  g_forced.clear();
  g_grouped.clear();
  g_grouped_forced.clear();
  g_batched.clear();
  g_batched_forced.clear();
  st_entries.store(0);
  return AC_OK;
}

adaptcore_status adaptcore_read_probe(const void* buf, int64_t bytes, void* sink, void* stream) {
  if (!buf || !sink || bytes < 0) return fail(AC_ERR_INVALID_VALUE, "bad argument");
  adaptcore_status st = ensure_init();
  if (st != AC_OK) return st;
  const hipError_t e = ac::launch_read_probe(buf, bytes, sink, static_cast<hipStream_t>(stream));
  if (e == hipErrorInvalidValue) return fail(AC_ERR_INVALID_VALUE, "buffer or size not 16-byte aligned");
  if (e != hipSuccess) return fail(AC_ERR_LAUNCH, std::string("kernel launch failed: ") + hipGetErrorString(e));
  return AC_OK;
}

adaptcore_status adaptcore_bench_lookup(int64_t n_keys, int64_t n_lookups, double* ns_per_lookup) {
  if (n_keys <= 0 || n_lookups <= 0 || !ns_per_lookup) return fail(AC_ERR_INVALID_VALUE, "bad argument");
  std::vector<std::tuple<int64_t, int64_t, int64_t>> keys;
  keys.reserve((size_t)n_keys);
  uint64_t x = 0x2545F4914F6CDD1Dull;
  for (int64_t i = 0; i < n_keys; ++i) {
    x ^= x << 13;
    x ^= x >> 7;
    x ^= x << 17;
    keys.emplace_back(1 + (int64_t)(x % 1000), 1 + (int64_t)((x >> 20) % 1000), 1 + (int64_t)((x >> 40) % 1000));
  }
  for (auto& k : keys)
    if (!lookup(std::get<0>(k), std::get<1>(k), std::get<2>(k), AC_BF16_BF16OUT, 0)) return AC_ERR_INTERNAL;
  const int64_t batch = std::max<int64_t>(1, std::min<int64_t>(n_lookups, 1000));
  std::vector<double> per;
  uintptr_t sink = 0;
  for (int64_t done = 0, i = 0; done < n_lookups; done += batch) {
    const auto t0 = std::chrono::steady_clock::now();
    for (int64_t j = 0; j < batch; ++j, i = (i + 1) % n_keys) {
      auto& k = keys[(size_t)i];
      sink += (uintptr_t)lookup(std::get<0>(k), std::get<1>(k), std::get<2>(k), AC_BF16_BF16OUT, 0);
    }
    per.push_back(std::chrono::duration<double, std::nano>(std::chrono::steady_clock::now() - t0).count() / batch);
  }
  std::sort(per.begin(), per.end());
  *ns_per_lookup = per[per.size() / 2] + (sink == 1 ? 1e-9 : 0.0);
  return AC_OK;
}

const char* adaptcore_last_error(void) { return t_err.c_str(); }

adaptcore_status adaptcore_last_status(void) { return t_status; }

adaptcore_status adaptcore_taxonomy(const adaptcore_taxonomy_in_t* in, adaptcore_taxonomy_out_t* out) {
  if (!in || !out) return fail(AC_ERR_INVALID_VALUE, "null argument");
  if (in->M <= 0 || in->N <= 0 || in->K <= 0 || in->m <= 0 || in->n <= 0 || in->k <= 0 || in->m1 <= 0 ||
      in->n1 <= 0 || in->k1 <= 0 || in->n_core <= 0 || in->s_acc <= 0)
    return fail(AC_ERR_INVALID_VALUE, "taxonomy parameters must be positive");
  ac::taxonomy(*in, out);
  return AC_OK;
}

int32_t adaptcore_config_index(int32_t family, int32_t cfg) { return ac::config_index(family, cfg); }

double adaptcore_schedule(int32_t kind, int64_t Q, int64_t L, double t_m, double t_p, double t_drain) {
  return ac::schedule(kind, Q, L, t_m, t_p, t_drain);
}

}  // extern "C"
