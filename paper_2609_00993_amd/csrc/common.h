// Device helpers shared by the libmoepd kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moepd {

constexpr int kWave = 64;

// ---- bfloat16 <-> float32 ---------------------------------------------------

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// Round to nearest, ties to even.  NaN stays NaN (quiet bit set).  Written
// without branches so that epilogues converting many values stay straight-line.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t rne = u + 0x7fffu + ((u >> 16) & 1u);
  const uint32_t r = ((u & 0x7fffffffu) > 0x7f800000u) ? (u | 0x00400000u) : rne;
  return uint16_t(r >> 16);
}

// ---- wave utilities ----------------------------------------------------------

__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// Wave-wide maximum / minimum of a 32-bit unsigned value, returned to all
// lanes (wave-uniform).  Register moves across lanes (DPP), not LDS-routed
// shuffles: swaps within quads, then rotations by 4 and 8 lanes give every
// lane its 16-lane row's extremum; two row broadcasts (lane 15 of rows 0
// and 2 into rows 1 and 3, then lane 31 into rows 2 and 3) leave the wave's
// on lane 63, which is read out.
template <bool MAX, int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_step(uint32_t v) {
  // lanes left out read the extremum's identity (0 / all ones)
  const uint32_t o = __builtin_amdgcn_update_dpp(MAX ? 0u : 0xffffffffu, v, CTRL, ROW_MASK, 0xF, false);
  return MAX ? (o > v ? o : v) : (o < v ? o : v);
}
template <bool MAX>
__device__ __forceinline__ uint32_t wave_extremum_u32(uint32_t v) {
  v = dpp_step<MAX, 0xB1, 0xF>(v);   // quad_perm [1,0,3,2]
  v = dpp_step<MAX, 0x4E, 0xF>(v);   // quad_perm [2,3,0,1]
  v = dpp_step<MAX, 0x124, 0xF>(v);  // row_ror:4
  v = dpp_step<MAX, 0x128, 0xF>(v);  // row_ror:8
  v = dpp_step<MAX, 0x142, 0xA>(v);  // row_bcast:15
  v = dpp_step<MAX, 0x143, 0xC>(v);  // row_bcast:31
  return __builtin_amdgcn_readlane(v, 63);
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) { return wave_extremum_u32<true>(v); }
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) { return wave_extremum_u32<false>(v); }

// Inclusive wave scan of int32.
__device__ __forceinline__ int wave_inclusive_scan(int v) {
  const int l = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    int o = __shfl_up(v, off, kWave);
    if (l >= off) v += o;
  }
  return v;
}

// ---- 16-byte vector type for row copies --------------------------------------

// A native clang vector (not HIP's union-based uint4) so that arrays of them
// stay in registers.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 load16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void store16(void* p, const u32x4& v) { *reinterpret_cast<u32x4*>(p) = v; }

}  // namespace moepd
