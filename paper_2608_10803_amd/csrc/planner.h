// Host-side planner: tiling taxonomy, candidate enumeration, legality and the
// analytical latency model. Pure C++ (no HIP), so it runs and is tested on a
// machine without a GPU.
#pragma once
#include <stdint.h>

#include <string>
#include <vector>

#include "adaptcore.h"
#include "kernel_args.h"
#include "variants.h"

namespace ac {

struct Shape {
  int64_t M, N, K;
  int dtype;  // adaptcore_dtype
  uint32_t layouts;
};

// A selected configuration and everything needed to launch it.
struct Plan {
  Shape s;
  uint64_t shape_key = 0, variant_key = 0;
  int cls = AC_CLASS_COMMON;  // taxonomy template of the shape
  int family = FAM_TILE, cfg = 0, swizzle = 0;
  int unal = 0;  // direct-to-LDS family: operand tiles loaded through registers (any alignment)
  int tile_m = 0, tile_n = 0, tile_k = 0;
  int pm = 0, pn = 0, pk = 1;
  int kper = 0;          // k-blocks per partition
  int grid_x = 0, grid_y = 1;
  int iters_per_wg = 0;  // stream-K
  int sk_tiles = 0;      // stream-K
  int ws_pk = 0;         // stream-K: partial slots per split tile
  int n_launch = 1;      // kernels per call (split K and stream-K add a reduction)
  int64_t ws_bytes = 0;  // fp32 partials, then the row-major copies of transposed operands
  // Prologue (Eq. 7's T_pro): byte offsets in the workspace of the row-major
  // copies of a column-major A (M x ld8(K)) and B (K x ld8(N)); -1: none.
  int64_t ws_a_off = -1, ws_b_off = -1;
  double t_pro = 0;      // its model time, included in `predicted`
  int n_candidates = 0;
  double predicted = 0;
  int64_t groups = 0;    // grouped product: groups (s.M is then the row capacity);
                         // strided batch: batch count (s is every batch's shape)
};

struct Candidate {
  Plan p;
};

// Default profile of one MI355X.
adaptcore_hw_t default_hw();

// Runtime occupancy (workgroups per CU) of a kernel configuration; the
// registry fills this in when a device is present.
void set_runtime_occupancy(int family, int cfg, int occ);
int occupancy(int family, int cfg);

// Taxonomy of the shape (Section 4.2, with the reading of Section 4.3 for
// the base tile): spatial sufficiency of the largest menu tile that
// saturates the CUs, accumulator fit of that tile.
int classify_shape(const Shape& s, const adaptcore_hw_t& hw, int* base_cfg);

// All legal candidates with their model latencies, best first. The
// taxonomy's template restricts the search unless hw.search_open is set.
std::vector<Plan> enumerate(const Shape& s, const adaptcore_hw_t& hw, int* cls_out);

// Fills launch fields and predicted latency for one configuration key;
// returns false if the key is not legal for the shape.
bool plan_for_key(const Shape& s, const adaptcore_hw_t& hw, uint64_t key, Plan* out);

// Grouped product of `groups` groups over a row capacity of s.M rows: the
// model's choice among the grouped tile configurations (plan_grouped), or
// one configuration forced by its key (grouped_for_key).
bool plan_grouped(const Shape& s, int64_t groups, const adaptcore_hw_t& hw, Plan* out);
bool grouped_for_key(const Shape& s, int64_t groups, const adaptcore_hw_t& hw, uint64_t key, Plan* out);

// Strided batch of `batch` products of shape s on the grouped kernel.
bool plan_batched(const Shape& s, int64_t batch, const adaptcore_hw_t& hw, Plan* out);
bool batched_for_key(const Shape& s, int64_t batch, const adaptcore_hw_t& hw, uint64_t key, Plan* out);

// 64-bit shape key: M | N << 17 | K << 34 | dtype << 51 | layouts << 55, for
// dimensions below 2^17; larger shapes set bit 63 and hash all fields.
uint64_t shape_key(const Shape& s, bool* exact);

// Kernels one call of the plan launches, ';'-separated (template arguments
// as a profiler prints them).
std::string kernel_names(const Plan& p);

// Index of a configuration in the calibrated cost tables of the profile.
int config_index(int family, int cfg);

// Paper arithmetic for explicit tiling parameters (adaptcore_taxonomy).
void taxonomy(const adaptcore_taxonomy_in_t& in, adaptcore_taxonomy_out_t* out);
double schedule(int kind, int64_t Q, int64_t L, double tm, double tp, double tdrain);

}  // namespace ac
