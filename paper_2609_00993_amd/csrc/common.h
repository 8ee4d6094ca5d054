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

// One step of a wave maximum over DPP: each lane in the rows ROW_MASK
// enables takes the larger of its key and the key DPP control CTRL names;
// the other lanes keep their own.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint64_t dpp_max_step(uint64_t v) {
  const uint32_t lo = uint32_t(v), hi = uint32_t(v >> 32);
  const uint32_t olo = __builtin_amdgcn_update_dpp(lo, lo, CTRL, ROW_MASK, 0xF, false);
  const uint32_t ohi = __builtin_amdgcn_update_dpp(hi, hi, CTRL, ROW_MASK, 0xF, false);
  const uint64_t o = (uint64_t(ohi) << 32) | olo;
  return o > v ? o : v;
}

// Wave-wide maximum of a 64-bit key, returned to all lanes.  Register moves
// across lanes (DPP) rather than LDS-routed shuffles, so the k selections
// of the top-k kernel are a short dependent chain: swaps within quads, then
// rotations by 4 and 8 lanes give every lane its 16-lane row's maximum; two
// row broadcasts (lane 15 of rows 0 and 2 into rows 1 and 3, then lane 31
// into rows 2 and 3) leave the wave's maximum on lane 63, which is read out.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
  v = dpp_max_step<0xB1, 0xF>(v);   // quad_perm [1,0,3,2]
  v = dpp_max_step<0x4E, 0xF>(v);   // quad_perm [2,3,0,1]
  v = dpp_max_step<0x124, 0xF>(v);  // row_ror:4
  v = dpp_max_step<0x128, 0xF>(v);  // row_ror:8
  v = dpp_max_step<0x142, 0xA>(v);  // row_bcast:15
  v = dpp_max_step<0x143, 0xC>(v);  // row_bcast:31
  const uint32_t lo = __builtin_amdgcn_readlane(uint32_t(v), 63);
  const uint32_t hi = __builtin_amdgcn_readlane(uint32_t(v >> 32), 63);
  return (uint64_t(hi) << 32) | lo;
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
