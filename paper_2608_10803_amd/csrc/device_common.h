// Device helpers shared by the gfx950 kernel files: vector types, the
// MFMA instructions and the 16-bit output rounding of the input format, the
// AddMM epilogue, the XCD-aware tile order and buffer-resource constants.
// Included INSIDE the kernels' namespace (ac, or ac::f16 when the file is
// compiled with AC_INPUT_F16=1), after hip_runtime.h and kernel_args.h.

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
#if AC_INPUT_F16
typedef _Float16 in16x8 __attribute__((ext_vector_type(8)));
#else
typedef __bf16 in16x8 __attribute__((ext_vector_type(8)));
#endif

// 16-byte load from a 2-byte aligned address. gfx950 runs in unaligned
// access mode, and the compiler emits one dwordx4 load for this copy.
__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  u32x4 v;
  __builtin_memcpy(&v, p, 16);
  return v;
}

// Drops the first s (0..8) 16-bit elements of v, shifting the rest down and
// filling with zeros. Branch-free (selects only).
__device__ __forceinline__ u32x4 shift_down(u32x4 v, int s) {
  const uint64_t lo = (uint64_t)v[0] | ((uint64_t)v[1] << 32);
  const uint64_t hi = (uint64_t)v[2] | ((uint64_t)v[3] << 32);
  const int sb = s * 16;  // 0 .. 128
  const int s1 = sb & 63;
  const uint64_t lo_a = (lo >> s1) | (s1 ? (hi << (64 - s1)) : 0ull);  // sb < 64
  const uint64_t hi_a = hi >> s1;
  const uint64_t lo_b = hi >> s1;                                       // 64 <= sb < 128
  const uint64_t nlo = sb < 64 ? lo_a : (sb < 128 ? lo_b : 0ull);
  const uint64_t nhi = sb < 64 ? hi_a : 0ull;
  return u32x4{(uint32_t)nlo, (uint32_t)(nlo >> 32), (uint32_t)nhi, (uint32_t)(nhi >> 32)};
}

// Elements e .. e+7 of a row of `len` >= 8 elements; those at index >= len
// read as zero. The 16-byte load ends at the row end at the latest, so it
// never leaves the row, and no lane branches (no waits inside branches).
__device__ __forceinline__ u32x4 load_row8(const uint16_t* row, int64_t e, int64_t len) {
  const int64_t start = min(e, len - 8);
  const int s = (int)min<int64_t>(e - start, 8);
  return shift_down(load16(row + start), s);
}

// The same for rows of fewer than 8 elements: eight 2-byte loads at clamped
// indices, then selects.
__device__ __forceinline__ u32x4 load_row8_small(const uint16_t* row, int64_t e, int64_t len) {
  uint32_t h[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int64_t idx = e + i;
    const uint32_t v = row[min(max(idx, (int64_t)0), len - 1)];
    h[i] = idx < len ? v : 0u;
  }
  return u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
}

// Elements e .. e+7 of a row of `len` >= 1 elements, zeros past the end.
__device__ __forceinline__ u32x4 load_row(const uint16_t* row, int64_t e, int64_t len) {
  return len >= 8 ? load_row8(row, e, len) : load_row8_small(row, e, len);
}

#if AC_INPUT_F16
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(in16x8, a), __builtin_bit_cast(in16x8, b), c, 0,
                                                0, 0);
}
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(in16x8, a), __builtin_bit_cast(in16x8, b), c, 0,
                                                0, 0);
}
// fp32 -> the 16-bit output format, round to nearest even; NaN stays NaN
__device__ __forceinline__ uint16_t to16(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }
// c + a.lo * b.lo + a.hi * b.hi for two packed pairs of inputs (v_dot2c_f32_f16)
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, a), __builtin_bit_cast(h2, b), c, false);
}
// the value of a 16-bit input element (low 16 bits of h)
__device__ __forceinline__ float from16(uint32_t h) { return (float)__builtin_bit_cast(_Float16, (uint16_t)h); }
#else
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(in16x8, a), __builtin_bit_cast(in16x8, b), c, 0,
                                                 0, 0);
}
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(in16x8, a), __builtin_bit_cast(in16x8, b), c, 0,
                                                 0, 0);
}
__device__ __forceinline__ uint16_t to16(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
// c + a.lo * b.lo + a.hi * b.hi for two packed pairs of inputs (v_dot2c_f32_bf16)
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(b2, a), __builtin_bit_cast(b2, b), c, false);
}
__device__ __forceinline__ float from16(uint32_t h) { return __uint_as_float(h << 16); }
#endif

template <bool OBF>
__device__ __forceinline__ void store_c(void* C, int64_t idx, float v) {
  if constexpr (OBF)
    static_cast<uint16_t*>(C)[idx] = to16(v);
  else
    static_cast<float*>(C)[idx] = v;
}

// ---- AddMM epilogue on outputs of one row (uniform test of g.epi; C_old is
// read only where an output exists and beta != 0)
template <bool OBF>
__device__ __forceinline__ float c_old(const GemmArgs& g, int64_t row, int64_t col) {
  if constexpr (OBF)
    return from16(static_cast<const uint16_t*>(g.C)[row * g.ldc + col]);
  else
    return static_cast<const float*>(g.C)[row * g.ldc + col];
}
template <bool OBF, int NV>
__device__ __forceinline__ void epi_apply(const GemmArgs& g, float (&v)[NV], int64_t row, int64_t col,
                                          int64_t valid) {
  if (!g.epi) return;
#pragma unroll
  for (int e = 0; e < NV; ++e) {
    if (e < valid) {
      float x = g.alpha * v[e];
      if (g.bias) x += g.bias[col + e];
      if (g.beta != 0.f) x += g.beta * c_old<OBF>(g, row, col + e);
      v[e] = x;
    }
  }
}

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

// Buffer resources (raw, 32-bit data): an offset past every range reads
// zero and drops stores.
constexpr int32_t OOB_OFF = (int32_t)0x80000000u;  // past every tile's range
constexpr uint32_t RSRC_WORD3 = 0x00020000u;      // raw buffer, 32-bit data

// ---- LDS pipelines fed by direct-to-LDS loads (buffer_load ... lds)
typedef __attribute__((address_space(3))) void lds_void;

// A stage: chunk c (8 k) of row r sits at slot c ^ swz_a(r) of the row's
// slots (8 for 64-deep, 4 for 32-deep blocks): the lanes that read 8 or 16
// consecutive rows at one chunk fall on distinct banks, for 32 as for 64
// banks.
template <int BK>
__device__ __forceinline__ int swz_a(int r) {
  if constexpr (BK == 64)
    return (r & 7) ^ ((r >> 3) & 1);
  else
    return ((r >> 1) & 3) ^ ((r >> 3) & 1);
}

// s_waitcnt immediate for vmcnt(n) alone (expcnt 7 and lgkmcnt 15 do not
// wait; vmcnt bits 3:0 and 15:14)
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
