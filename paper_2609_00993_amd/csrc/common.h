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

// Wave-wide maximum of a 64-bit key, all lanes receive the result.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    uint32_t lo = __shfl_xor(uint32_t(v), off, kWave);
    uint32_t hi = __shfl_xor(uint32_t(v >> 32), off, kWave);
    uint64_t o = (uint64_t(hi) << 32) | lo;
    v = o > v ? o : v;
  }
  return v;
}

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
