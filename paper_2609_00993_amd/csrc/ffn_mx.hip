// FP8 expert layer on CDNA4's MX-scaled matrix cores: OCP MX FP8 operands
// (E4M3 codes, one E8M0 scale per 32 consecutive values along K), float32
// accumulation.  The paper runs BF16 and FP8 checkpoints of its model
// (Section 7.1) without describing the FP8 format; MX FP8 is the format the
// gfx950 matrix cores scale natively.
//
//  * permute_mx: the dispatch data movement of an FP8 context quantizes each
//    token's bf16 row once (per 32 values: shared exponent E = floor(log2
//    amax) - 8, codes = RNE(clamp(v / 2^E, +-448))) and writes the codes and
//    scale bytes to every row the token occupies;
//  * GEMM1 / GEMM2: v_mfma_scale_f32_32x32x64_f8f6f4 over 64-deep K steps.
//    Lane l of an operand holds row l % 32: its bytes 0-15 are K [16h, 16h+16)
//    and bytes 16-31 are K [32 + 16h, +16) of the step (h = l / 32), and its
//    scale register carries the scale of K block h of the step (32 values)
//    for that row.  GEMM1's epilogue applies the SwiGLU and quantizes h per
//    32 columns of a row (the two lanes holding a row's 32 columns exchange
//    their maxima), GEMM2 writes float32 y.
//
// The GEMM here is the weight-streaming tile (32 rows x 128 columns, each
// wave reading its operand rows straight into registers), which every batch
// size uses.
#include "common.h"
#include "kernels.h"
#include "tiles.h"

namespace moepd {

typedef int32_t v8i32 __attribute__((ext_vector_type(8)));
typedef float f32x16_mx __attribute__((ext_vector_type(16)));
typedef float f32x4_mx __attribute__((ext_vector_type(4)));

constexpr float kE4M3Max = 448.f;

// Shared exponent of a block from its largest magnitude: floor(log2 amax) - 8
// from the float's exponent field (amax = 0 or subnormal gives -127; a
// normal amax never gives more than 119).
__device__ __forceinline__ int mx_exponent(float amax) {
  const int ef = (int)((__float_as_uint(amax) >> 23) & 0xffu);
  const int e = ef - 127 - 8;
  return ef == 0 ? -127 : (e < -127 ? -127 : e);
}

// 2^-e as a float for e in [-127, 119]: exact powers of two (2^127 at most).
__device__ __forceinline__ float pow2_neg(int e) { return ldexpf(1.f, -e); }

// Two values (already scaled) to two E4M3 codes, packed into the low half
// of the result (RNE; the clamp makes |v| <= 448 so nothing overflows).
__device__ __forceinline__ uint32_t e4m3_pair(float a, float b) {
  a = fminf(fmaxf(a, -kE4M3Max), kE4M3Max);
  b = fminf(fmaxf(b, -kE4M3Max), kE4M3Max);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false) & 0xffffu;
}

// ------------------------------------------------------------------ permute + quantize

// One wave per token.  Lane l takes 16-byte vector v = v0 + l of the bf16 row
// (8 values); four consecutive lanes hold one 32-value block.
__global__ __launch_bounds__(256) void permute_mx_kernel(const u32x4* __restrict__ x, int T, int k, int H,
                                                         const int32_t* __restrict__ row_of_slot,
                                                         uint8_t* __restrict__ codes, uint8_t* __restrict__ scales) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;  // whole wave leaves together
  const int lane = threadIdx.x & 63;
  const int r_l = lane < k ? row_of_slot[(size_t)t * k + lane] : -1;
  const uint64_t resident = __ballot(r_l >= 0);
  if (!resident) return;
  const int nv = H / 8, nb = H / 32;
  const u32x4* xt = x + (size_t)t * nv;
  for (int v0 = 0; v0 < nv; v0 += kWave) {
    const int v = v0 + lane;
    const bool on = v < nv;  // nv is a multiple of 4: a block is all on or all off
    float f[8];
    float amax = 0.f;
    if (on) {
      const u32x4 u = xt[v];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f[2 * i] = __uint_as_float(u[i] << 16);
        f[2 * i + 1] = __uint_as_float(u[i] & 0xffff0000u);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(f[i]));
    }
    amax = fmaxf(amax, __shfl_xor(amax, 1, kWave));
    amax = fmaxf(amax, __shfl_xor(amax, 2, kWave));
    const int e = mx_exponent(amax);
    const float inv = pow2_neg(e);
    uint32_t lo = 0, hi = 0;
    if (on) {
      lo = e4m3_pair(f[0] * inv, f[1] * inv) | (e4m3_pair(f[2] * inv, f[3] * inv) << 16);
      hi = e4m3_pair(f[4] * inv, f[5] * inv) | (e4m3_pair(f[6] * inv, f[7] * inv) << 16);
    }
    uint64_t m = resident;
    while (m) {
      const int j = __builtin_ctzll(m);
      m &= m - 1;
      const int row = __builtin_amdgcn_readlane(r_l, j);
      if (on) {
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        *reinterpret_cast<u32x2*>(codes + (size_t)row * H + (size_t)v * 8) = u32x2{lo, hi};
        if ((lane & 3) == 0) scales[(size_t)row * nb + v / 4] = (uint8_t)(e + 127);
      }
    }
  }
}

hipError_t launch_permute_mx(const void* x, int T, int k, int H, const int32_t* row_of_slot, uint8_t* codes,
                             uint8_t* scales, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  permute_mx_kernel<<<dim3((T + 3) / 4), dim3(256), 0, s>>>((const u32x4*)x, T, k, H, row_of_slot, codes, scales);
  return hipGetLastError();
}

// ------------------------------------------------------------------ grouped GEMM

struct GemmArgsMX {
  const uint8_t* A;   // [R, K] codes, expert-contiguous rows
  const uint8_t* As;  // [R, K / 32] scales
  const uint8_t* B;   // expert e at B + e * b_stride: [N rows (x2 for gate/up), K] codes
  const uint8_t* Bs;  // expert e at Bs + e * bs_stride: [rows, K / 32] scales
  void* C;            // GATED: h codes [R, N]; else float32 y [R, N]
  uint8_t* Cs;        // GATED: h scales [R, N / 32]
  const int32_t* offsets;
  const int32_t* tile_base;
  long long b_stride, bs_stride;
  int e_loc, N, K, n_tiles, up_row;
  int n_group, xcd_local;
  YieldTo yield;
};

__device__ __forceinline__ v8i32 join(const u32x4& a, const u32x4& b) {
  return v8i32{(int32_t)a[0], (int32_t)a[1], (int32_t)a[2], (int32_t)a[3],
               (int32_t)b[0], (int32_t)b[1], (int32_t)b[2], (int32_t)b[3]};
}

// silu(g) * u (the hardware reciprocal, about 1 ulp, is far inside E4M3's
// rounding of h).
__device__ __forceinline__ float silu_mul_mx(float gt, float up) {
  return gt * __builtin_amdgcn_rcpf(1.f + __expf(-gt)) * up;
}

// One wave: 32 output columns x 32 rows of the tile, over all of K.  The
// MFMAs take the weight rows as their first operand, so lane l ends with
// token row l % 32 and the 16 columns 8q + 4h + (0..3), q = 0..3.
template <bool GATED>
__device__ __forceinline__ void gemm_mx_skinny_tile(const GemmArgsMX& g, const TileCoord& tc) {
  constexpr int NB = GATED ? 2 : 1;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 31, h = lane >> 5;
  const int col0 = tc.n0 + wave * 32;
  if (col0 >= g.N) return;  // N is a multiple of 32: a wave's columns are all in or all out
  const int arow = min(tc.m0 + r, tc.m_end - 1);
  const int wrow = col0 + r;
  const int KS = g.K / 32;
  const uint8_t* Be = g.B + (size_t)tc.e * g.b_stride;
  const uint8_t* Bse = g.Bs + (size_t)tc.e * g.bs_stride;
  // 16-byte units of a row; a 128-deep K block is 8 units, the lane takes
  // units 2p + h of each 64-deep step (p = 0, 1)
  const u32x4* pa = reinterpret_cast<const u32x4*>(g.A + (size_t)arow * g.K) + h;
  const uint8_t* psa = g.As + (size_t)arow * KS + h;
  const u32x4* pb[NB];
  const uint8_t* psb[NB];
  pb[0] = reinterpret_cast<const u32x4*>(Be + (size_t)wrow * g.K) + h;
  psb[0] = Bse + (size_t)wrow * KS + h;
  if (GATED) {
    pb[NB - 1] = reinterpret_cast<const u32x4*>(Be + (size_t)(g.up_row + wrow) * g.K) + h;
    psb[NB - 1] = Bse + (size_t)(g.up_row + wrow) * KS + h;
  }

  f32x16_mx acc[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[j][q] = 0.f;

  const int KB = g.K / 128;
  constexpr int PF = 2;  // 128-deep K blocks in flight per wave
  u32x4 ra[PF][4], rb[PF][NB][4];
  int sa[PF][2], sb[PF][NB][2];
  auto load = [&](int kb, u32x4 (&a)[4], u32x4 (&b)[NB][4], int (&ssa)[2], int (&ssb)[NB][2]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      a[u] = pa[kb * 8 + 2 * u];
#pragma unroll
      for (int j = 0; j < NB; ++j) b[j][u] = pb[j][kb * 8 + 2 * u];
    }
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      ssa[s] = psa[kb * 4 + 2 * s];
#pragma unroll
      for (int j = 0; j < NB; ++j) ssb[j][s] = psb[j][kb * 4 + 2 * s];
    }
  };
#pragma unroll
  for (int p = 0; p < PF; ++p)
    if (p < KB) load(p, ra[p], rb[p], sa[p], sb[p]);
  for (int kb0 = 0; kb0 < KB; kb0 += PF) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int kb = kb0 + p;
      if (kb < KB) {
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
          for (int j = 0; j < NB; ++j)
            acc[j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                join(rb[p][j][2 * s], rb[p][j][2 * s + 1]), join(ra[p][2 * s], ra[p][2 * s + 1]), acc[j], 0, 0, 0,
                sb[p][j][s], 0, sa[p][s]);
        if (kb + PF < KB) load(kb + PF, ra[p], rb[p], sa[p], sb[p]);
      }
    }
  }

  const int row = tc.m0 + r;
  if (row >= tc.m_end) return;
  if (GATED) {
    float v[16];
    float amax = 0.f;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      v[q] = silu_mul_mx(acc[0][q], acc[NB - 1][q]);
      amax = fmaxf(amax, fabsf(v[q]));
    }
    amax = fmaxf(amax, __shfl_xor(amax, 32, kWave));  // the row's other 16 columns
    const int e = mx_exponent(amax);
    const float inv = pow2_neg(e);
    uint8_t* hrow = static_cast<uint8_t*>(g.C) + (size_t)row * g.N + col0 + 4 * h;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t w = e4m3_pair(v[4 * q] * inv, v[4 * q + 1] * inv) |
                         (e4m3_pair(v[4 * q + 2] * inv, v[4 * q + 3] * inv) << 16);
      *reinterpret_cast<uint32_t*>(hrow + 8 * q) = w;
    }
    if (h == 0) g.Cs[(size_t)row * (g.N / 32) + col0 / 32] = (uint8_t)(e + 127);
  } else {
    float* yrow = static_cast<float*>(g.C) + (size_t)row * g.N + col0 + 4 * h;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<f32x4_mx*>(yrow + 8 * q) =
          f32x4_mx{acc[0][4 * q], acc[0][4 * q + 1], acc[0][4 * q + 2], acc[0][4 * q + 3]};
  }
}

template <bool GATED>
__global__ __launch_bounds__(256) void gemm_mx_skinny(GemmArgsMX g) {
  const int L = block_tile(g);
  if (L < 0) return;
  yield_to_window(g.yield);
  TileCoord tc;
  tile_at(g, L, 32, 128, tc);
  gemm_mx_skinny_tile<GATED>(g, tc);
}

static inline int round8_mx(long long v) { return (int)((v + 7) / 8 * 8); }

hipError_t launch_ffn_mx(int gemm, const PhaseBuffers& b, const MxBuffers& mx, const MxWeights& w, int e_loc, int H,
                         int I, int max_m_tiles, YieldTo yield, hipStream_t s) {
  GemmArgsMX g{};
  g.offsets = b.offsets;
  g.tile_base = b.tile_base;
  g.e_loc = e_loc;
  g.yield = yield;
  g.n_group = 1;
  g.xcd_local = 1;
  if (gemm == 1) {
    g.A = mx.x_codes;
    g.As = mx.x_scales;
    g.B = (const uint8_t*)w.gu;
    g.Bs = (const uint8_t*)w.gu_scales;
    g.C = mx.h_codes;
    g.Cs = mx.h_scales;
    g.b_stride = 2LL * I * H;
    g.bs_stride = 2LL * I * (H / 32);
    g.N = I;
    g.K = H;
    g.up_row = I;
  } else {
    g.A = mx.h_codes;
    g.As = mx.h_scales;
    g.B = (const uint8_t*)w.dn;
    g.Bs = (const uint8_t*)w.dn_scales;
    g.C = b.y;
    g.Cs = nullptr;
    g.b_stride = (long long)H * I;
    g.bs_stride = (long long)H * (I / 32);
    g.N = H;
    g.K = I;
    g.up_row = 0;
  }
  g.n_tiles = (g.N + 127) / 128;
  const dim3 grid(round8_mx((long long)max_m_tiles * g.n_tiles));
  if (gemm == 1) gemm_mx_skinny<true><<<grid, 256, 0, s>>>(g);
  else gemm_mx_skinny<false><<<grid, 256, 0, s>>>(g);
  return hipGetLastError();
}

int ffn_mx_bm() { return 32; }

}  // namespace moepd
