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
