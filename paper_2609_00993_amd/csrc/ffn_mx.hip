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
// Two tile shapes, as in the bf16 layer: the weight-streaming tile for small
// batches (32 rows x 32 columns, one wave per workgroup, operands through
// the wave's LDS stage) and, for large batches, 256 x 128 (gate + up) /
// 256 x 256 tiles staged through a two-slot LDS ring of 128-deep K slices
// (128 bytes per row, the byte layout of the bf16 ring's 64-deep slices),
// with the slices' scale bytes staged alongside.  256-row tiles read an
// expert of up to 256 rows' weights once; against 128-row tiles in a
// three-slot ring they took the 8192-token layer's GEMM1 from 445 to 392 us.
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "pipeline.h"
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

// One wave per token (per part of its row for small batches, see
// waves_per_row).  Lane l takes 16-byte vector v = v0 + l of the bf16 row
// (8 values); four consecutive lanes hold one 32-value block.
__global__ __launch_bounds__(256) void permute_mx_kernel(const u32x4* __restrict__ x, int T, int k, int H,
                                                         int parts, const int32_t* __restrict__ row_of_slot,
                                                         uint8_t* __restrict__ codes, uint8_t* __restrict__ scales) {
  const int wi = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int t = wi / parts, part = wi - t * parts;
  if (t >= T) return;  // whole wave leaves together
  const int lane = threadIdx.x & 63;
  const int r_l = lane < k ? row_of_slot[(size_t)t * k + lane] : -1;
  const uint64_t resident = __ballot(r_l >= 0);
  if (!resident) return;
  const int nv = H / 8, nb = H / 32;
  const u32x4* xt = x + (size_t)t * nv;
  for (int v0 = part * kWave; v0 < nv; v0 += parts * kWave) {
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
  const int parts = waves_per_row(T, H / 8, 1);
  const long long waves = (long long)T * parts;
  permute_mx_kernel<<<dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s>>>((const u32x4*)x, T, k, H, parts,
                                                                             row_of_slot, codes, scales);
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
  int n_group, m_super, xcd_local;
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

// Small batches: one wave (32 output columns) per workgroup, so that the
// tiles spread evenly over the CUs whatever their count (with four-wave
// workgroups, 1.5 tiles per CU left half the CUs with two).
constexpr int kMxDecodeWaves = 1;

// One wave: 32 output columns x 32 rows of the tile, over all of K.  The
// MFMAs take the weight rows as their first operand, so lane l ends with
// token row l % 32 and the 16 columns 8q + 4h + (0..3), q = 0..3.
// A 128-deep K block of a panel (the tile's 32 code rows, or its 32 gate or
// up weight rows) is 4 KB: it is loaded by four 1 KB whole-line reads (lane
// l: row 8i + l/8, 16-byte unit l%8), written to this wave's LDS stage (unit
// c of row r at slot 8r + (c ^ stage_swz(r)), no bank conflicts either way) and read
// back in the MFMA lane layout; reading 16 bytes from each of 32 rows per
// instruction reaches only about a quarter of the per-CU rate of whole-line
// reads.  A row's four scale bytes of the block come as one 4-byte load.
// SC2 (K a multiple of 256, scale arrays 8-byte aligned): a row's scale
// bytes of two blocks come as one 8-byte load every second block.  Scale
// loads read a few bytes from each of 32 rows per instruction (the slow
// pattern), so halving them leaves the whole-line code loads more room.
template <bool GATED, bool SC2>
__device__ __forceinline__ void gemm_mx_skinny_tile(const GemmArgsMX& g, const TileCoord& tc) {
  static_assert(kMxDecodeWaves == 1, "the LDS stage below is private to the workgroup's one wave");
  constexpr int NB = GATED ? 2 : 1;
  constexpr int NP = 1 + NB;  // panels: code rows, then weight rows (gate, up)
  __shared__ u32x4 stage[NP][32 * 8];
  const int lane = threadIdx.x & 63;
  const int r = lane & 31, h = lane >> 5;
  const int lr = lane >> 3, lc = lane & 7;
  const int col0 = tc.n0;
  if (col0 >= g.N) return;  // N is a multiple of 32: a wave's columns are all in or all out
  const int KS = g.K / 32;
  const uint8_t* Be = g.B + (size_t)tc.e * g.b_stride;
  const uint8_t* Bse = g.Bs + (size_t)tc.e * g.bs_stride;
  const u32x4* base[NP];
  const uint32_t* sbase[NP];
  base[0] = reinterpret_cast<const u32x4*>(g.A);
  sbase[0] = reinterpret_cast<const uint32_t*>(g.As);
  base[1] = reinterpret_cast<const u32x4*>(Be);
  sbase[1] = reinterpret_cast<const uint32_t*>(Bse);
  if (GATED) {
    base[NP - 1] = reinterpret_cast<const u32x4*>(Be + (size_t)g.up_row * g.K);
    sbase[NP - 1] = reinterpret_cast<const uint32_t*>(Bse + (size_t)g.up_row * KS);
  }
  // Offsets in 16-byte units and scale words; 32 bits suffice (fewer than
  // 32 x 1024 code rows of at most 1024 units in this regime, at most
  // 2 x 16384 weight rows).
  const int kv = g.K / 16, kw = KS / 4;
  int off[NP][4], soff[NP];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int rr = 8 * i + lr;
    off[0][i] = min(tc.m0 + rr, tc.m_end - 1) * kv + lc;
#pragma unroll
    for (int j = 0; j < NB; ++j) off[1 + j][i] = (col0 + rr) * kv + lc;
  }
  soff[0] = min(tc.m0 + r, tc.m_end - 1) * kw;
#pragma unroll
  for (int j = 0; j < NB; ++j) soff[1 + j] = (col0 + r) * kw;
  int wslot[4];  // LDS slot of this lane's chunk for each of the four instructions
#pragma unroll
  for (int i = 0; i < 4; ++i) wslot[i] = (8 * i + lr) * 8 + (lc ^ stage_swz(8 * i + lr));
  // Step s (64 deep) of a block: lane (r, h) holds units 4s + h and 4s + 2 + h
  // of its row and the scale of 32-value block 2s + h.
  int rslot[2][2];
#pragma unroll
  for (int st = 0; st < 2; ++st)
#pragma unroll
    for (int u = 0; u < 2; ++u) rslot[st][u] = r * 8 + ((4 * st + 2 * u + h) ^ stage_swz(r));

  f32x16_mx acc[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[j][q] = 0.f;

  const int KB = g.K / 128;
  constexpr int PF = 2;  // 128-deep K blocks in flight per wave
  u32x4 v[PF][NP][4];
  auto mfma_block = [&](const uint32_t (&scl)[NP]) {
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const v8i32 a = join(stage[0][rslot[st][0]], stage[0][rslot[st][1]]);
      const int sa = (int)((scl[0] >> (16 * st)) & 0xffu);
#pragma unroll
      for (int j = 0; j < NB; ++j)
        acc[j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            join(stage[1 + j][rslot[st][0]], stage[1 + j][rslot[st][1]]), a, acc[j], 0, 0, 0,
            (int)((scl[1 + j] >> (16 * st)) & 0xffu), 0, sa);
    }
  };
  // LDS operations of one wave run in order, so a block's stage writes land
  // after the previous block's reads and before its own.
  auto stage_block = [&](const u32x4 (&d)[NP][4]) {
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int i = 0; i < 4; ++i) stage[p][wslot[i]] = d[p][i];
  };
  // Scale words of the block pair in flight (SC2) or of each block.
  typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
  uint32_t sc[PF][NP];
  u32x2 sp[NP], sp_next[NP];
  auto load = [&](int kb, u32x4 (&d)[NP][4], uint32_t (&ds)[NP]) {
#pragma unroll
    for (int p = 0; p < NP; ++p) {
#pragma unroll
      for (int i = 0; i < 4; ++i) d[p][i] = base[p][off[p][i] + kb * 8];
      if (SC2) {
        if ((kb & 1) == 0) sp_next[p] = *reinterpret_cast<const u32x2*>(sbase[p] + soff[p] + kb);
      } else {
        ds[p] = sbase[p][soff[p] + kb];
      }
    }
  };
#pragma unroll
  for (int q = 0; q < PF; ++q)
    if (q < KB) load(q, v[q], sc[q]);
  for (int kb0 = 0; kb0 < KB; kb0 += PF) {
    if (SC2) {
#pragma unroll
      for (int p = 0; p < NP; ++p) sp[p] = sp_next[p];
    }
#pragma unroll
    for (int q = 0; q < PF; ++q) {
      const int kb = kb0 + q;
      if (kb < KB) {
        stage_block(v[q]);
        uint32_t scl[NP];
#pragma unroll
        for (int p = 0; p < NP; ++p) scl[p] = (SC2 ? sp[p][q] : sc[q][p]) >> (8 * h);
        if (kb + PF < KB) load(kb + PF, v[q], sc[q]);
        mfma_block(scl);
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

// ------------------------------------------------------------------ LDS ring (prefill)

// One workgroup of 4 waves, a BM x BN output tile of one expert.  Per
// 128-deep K slice, A (BM rows) and B (BR = NB x BN weight rows) travel HBM ->
// LDS by 16-byte DMA into a ring of STAGES slots (swizzled like the bf16
// ring), and each row's four scale bytes of the slice (one per 32 values) by
// 4-byte DMA into the slot's scale area.  Every wave issues the same number
// of DMA instructions per slice (padding with a repeat of an A-scale gather
// into a spare area), so vmcnt counts retire exactly whole slices.  A slice
// is two 64-deep MFMA steps; fragments of the next step are read from LDS
// while the current step's MFMAs run.
template <int BM, int BR, int WM, int WN, bool GATED, int STAGES>
__device__ __forceinline__ void gemm_mx_ring_body(const GemmArgsMX& g) {
  constexpr int NB = GATED ? 2 : 1;
  constexpr int BN = BR / NB;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 32, FN = WTN / 32, FB = FN * NB;
  constexpr int BK = 128;                           // K values (bytes) per slice
  constexpr int CPR = 8;                            // 16-byte chunks per staged row
  constexpr int RPI = 8;                            // rows per 16-byte DMA instruction
  constexpr int A_INS = BM / RPI / 4, B_INS = BR / RPI / 4;
  constexpr int SC_ALL = (BM + BR) / 64;            // 4-byte gathers of scale rows per slice
  constexpr int SC_INS = (SC_ALL + 3) / 4;          // per wave, padded
  constexpr int NPS = A_INS + B_INS + SC_INS;       // vector-memory ops per wave per slice
  constexpr int A_CH = BM * CPR, B_CH = BR * CPR;
  constexpr int SC_W = BM + BR + 64;                // scale words per slot (+ spare for padding)
  constexpr int NRD = 2 * (FM + FB), NMF = FM * FB;
  static_assert(WM * WN == 4, "four waves");
  static_assert(A_INS * RPI * 4 == BM && B_INS * RPI * 4 == BR, "slices split into whole DMA instructions");
  static_assert(BM % 64 == 0 && BR % 64 == 0, "scale gathers of 64 rows");
  static_assert(FM * 32 == WTM && FN * 32 == WTN, "wave tile must be a multiple of 32x32");
  static_assert(STAGES >= 2 && NPS * (STAGES - 1) < 64, "pipeline depth");
  // each slot: A chunks, B chunks, then SC_W scale words (one array, so the
  // compiler sees the DMA'd scale words and the ring as one object)
  __shared__ u32x4 ring[STAGES][A_CH + B_CH + SC_W / 4];

  const int lane = threadIdx.x & 63;
  const int h = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int KT = g.K / BK;
  const int KS = g.K / 32;  // scale bytes per row
  const int lrow = lane / CPR, lphys = lane % CPR;

  __amdgpu_buffer_rsrc_t a_rsrc;
  uint32_t a_off[A_INS];
  const uint8_t* b_src[B_INS];
  const uint8_t* sc_src[SC_INS];  // this lane's scale word of slice 0 (rows clamped into range)
  int sc_dst[SC_INS];             // its 64-word group in the slot's scale area
  auto set_sources = [&](const TileCoord& tc) {
    const int m0 = __builtin_amdgcn_readfirstlane(tc.m0);
    const int rows = min(__builtin_amdgcn_readfirstlane(tc.m_end) - m0, BM);
    a_rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)(g.A + (size_t)m0 * g.K), (short)0, rows * g.K,
                                               kBufferRsrcWord3);
    const int e = __builtin_amdgcn_readfirstlane(tc.e);
    const uint8_t* Be = g.B + (size_t)e * g.b_stride;
    const uint8_t* Bse = g.Bs + (size_t)e * g.bs_stride;
#pragma unroll
    for (int i = 0; i < A_INS; ++i) {
      const int r = (wave * A_INS + i) * RPI + lrow;
      a_off[i] = (uint32_t)(r * g.K + (lphys ^ swz<64>(r)) * 16);
    }
    auto brow_of = [&](int r) {
      if (GATED) return r < BN ? min(tc.n0 + r, g.N - 1) : g.up_row + min(tc.n0 + r - BN, g.N - 1);
      return min(tc.n0 + r, g.N - 1);
    };
#pragma unroll
    for (int i = 0; i < B_INS; ++i) {
      const int r = (wave * B_INS + i) * RPI + lrow;
      b_src[i] = Be + (size_t)brow_of(r) * g.K + (lphys ^ swz<64>(r)) * 16;
    }
    // Every gather is the same instruction (no branch in the K loop): A-scale
    // rows past the expert's end are clamped to its last row (their outputs
    // are never stored); padding gathers repeat rows 0..63 into the spare area.
#pragma unroll
    for (int i = 0; i < SC_INS; ++i) {
      const int q = wave * SC_INS + i;
      const int qq = q < SC_ALL ? q : 0;
      const int r = qq * 64 + lane;
      if (r < BM) sc_src[i] = g.As + (size_t)min(m0 + r, tc.m_end - 1) * KS;
      else sc_src[i] = Bse + (size_t)brow_of(r - BM) * KS;
      sc_dst[i] = __builtin_amdgcn_readfirstlane(q < SC_ALL ? q * 64 : BM + BR);
    }
  };
  auto issue = [&](int kt, int slot) {
#pragma unroll
    for (int i = 0; i < A_INS; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(a_rsrc, MOEPD_LPTR(&ring[slot][(wave * A_INS + i) * 64]), 16,
                                               a_off[i] + (uint32_t)kt * BK, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < B_INS; ++i)
      __builtin_amdgcn_global_load_lds(MOEPD_GPTR(b_src[i] + kt * BK),
                                       MOEPD_LPTR(&ring[slot][A_CH + (wave * B_INS + i) * 64]), 16, 0, 0);
#pragma unroll
    for (int i = 0; i < SC_INS; ++i)
      __builtin_amdgcn_global_load_lds(MOEPD_GPTR(sc_src[i] + kt * 4),
                                       MOEPD_LPTR(&ring[slot][A_CH + B_CH + sc_dst[i] / 4]), 4, 0, 0);
  };
  auto prologue = [&](const TileCoord& tc) {
    set_sources(tc);
#pragma unroll
    for (int st = 0; st < STAGES; ++st)
      if (st < KT) issue(st, st);
  };

  // step s of a slice: lane half h takes chunks 4s + h and 4s + 2 + h of its
  // row (K [64s + 16h, +16) and [64s + 32 + 16h, +16)); its scale word holds
  // the slice's four block scales, of which step s uses byte 2s + h.
  v8i32 fa[2][FM], fb[2][FB];
  u32x4 sa_raw[FM], sb_raw[FB];
  uint32_t sa[FM], sb[FB];
  auto read_frags = [&](int slot, int sub, v8i32 (&a)[FM], v8i32 (&b)[FB]) {
    const u32x4* As = &ring[slot][0];
    const u32x4* Bs = &ring[slot][A_CH];
    const int c0 = 4 * sub + h, c1 = 4 * sub + 2 + h;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int r = wm * WTM + fm * 32 + (lane & 31);
      a[fm] = join(As[r * CPR + (c0 ^ swz<64>(r))], As[r * CPR + (c1 ^ swz<64>(r))]);
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        const int r = nb * BN + wn * WTN + fn * 32 + (lane & 31);
        b[nb * FN + fn] = join(Bs[r * CPR + (c0 ^ swz<64>(r))], Bs[r * CPR + (c1 ^ swz<64>(r))]);
      }
  };
  // Scale words are read as whole 16-byte groups (4-byte LDS reads right
  // after the DMA issue made the compiler wait for every outstanding DMA,
  // vmcnt(0), in the K loop); the lane's word is picked when the slice
  // starts, so the reads have the previous step's MFMAs to land.
  auto read_scales = [&](int slot, u32x4 (&ra)[FM], u32x4 (&rb)[FB]) {
    const u32x4* S = &ring[slot][A_CH + B_CH];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) ra[fm] = S[(wm * WTM + fm * 32 + (lane & 31)) >> 2];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) rb[nb * FN + fn] = S[(BM + nb * BN + wn * WTN + fn * 32 + (lane & 31)) >> 2];
  };
  auto pick = [&](const u32x4& v) {  // the lane's word (rows are multiples of 4 apart), shifted to block h
    const int c = lane & 3;
    const uint32_t w = c == 0 ? v[0] : c == 1 ? v[1] : c == 2 ? v[2] : v[3];
    return w >> (8 * h);
  };

  f32x16_mx acc[FM][FB];
  auto mfmas = [&](int sub, const v8i32 (&a)[FM], const v8i32 (&b)[FB]) {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int j = 0; j < FB; ++j)
        acc[fm][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(b[j], a[fm], acc[fm][j], 0, 0, 0,
                                                                     (int)(sb[j] >> (16 * sub)), 0,
                                                                     (int)(sa[fm] >> (16 * sub)));
  };

  const int L = block_tile(g);
  if (L < 0) return;
  yield_to_window(g.yield);
  TileCoord tc;
  tile_at(g, L, BM, BN, tc);
  prologue(tc);

#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FB; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  wait_slices_lgkm0<NPS, STAGES - 1>(min(STAGES - 1, KT - 1));
  bare_barrier();
  read_frags(0, 0, fa[0], fb[0]);
  read_scales(0, sa_raw, sb_raw);

  // One K slice (MODE as in the bf16 ring: 0 refills the slot, 1 has nothing
  // left to issue, 2 is the last slice).
  auto slice = [&](auto mode, int kt, int slot) {
    constexpr int MODE = decltype(mode)::value;
#pragma unroll
    for (int i = 0; i < FM; ++i) sa[i] = pick(sa_raw[i]);
#pragma unroll
    for (int j = 0; j < FB; ++j) sb[j] = pick(sb_raw[j]);
    // step 0: read step 1's fragments, multiply step 0
    read_frags(slot, 1, fa[1], fb[1]);
    mfmas(0, fa[0], fb[0]);
    interleave<0, NMF, 0, NRD, 0>();
    if constexpr (MODE < 2) {
      if constexpr (MODE == 0) wait_vmcnt_lgkm0<NPS * (STAGES - 2)>();
      else wait_slices_lgkm0<NPS, STAGES - 2>(min(STAGES - 2, KT - 2 - kt));
      bare_barrier();
      int ns = slot + 1;
      if (ns == STAGES) ns = 0;
      if constexpr (MODE == 0) issue(kt + STAGES, slot);
      read_frags(ns, 0, fa[0], fb[0]);
      read_scales(ns, sa_raw, sb_raw);
      mfmas(1, fa[1], fb[1]);
      interleave<0, NMF, MODE == 0 ? NPS : 0, NRD + FM + FB, 1>();
    } else {
      mfmas(1, fa[1], fb[1]);
    }
  };
  int kt = 0, slot = 0;
  for (; kt < KT - STAGES; ++kt) {
    slice(std::integral_constant<int, 0>{}, kt, slot);
    if (++slot == STAGES) slot = 0;
  }
  for (; kt < KT - 1; ++kt) {
    slice(std::integral_constant<int, 1>{}, kt, slot);
    if (++slot == STAGES) slot = 0;
  }
  slice(std::integral_constant<int, 2>{}, kt, slot);

  // epilogue (lane l: row l & 31 of each 32-row block, columns 8q + 4h + t)
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int row = tc.m0 + wm * WTM + fm * 32 + (lane & 31);
    const bool live = row < tc.m_end;
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int col0 = tc.n0 + wn * WTN + fn * 32;  // a 32-column block: all in range or all out
      if (GATED) {
        float v[16];
        float amax = 0.f;
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          v[q] = silu_mul_mx(acc[fm][fn][q], acc[fm][FN + fn][q]);
          amax = fmaxf(amax, fabsf(v[q]));
        }
        amax = fmaxf(amax, __shfl_xor(amax, 32, kWave));
        if (!live || col0 >= g.N) continue;
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
        if (!live || col0 >= g.N) continue;
        float* yrow = static_cast<float*>(g.C) + (size_t)row * g.N + col0 + 4 * h;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<f32x4_mx*>(yrow + 8 * q) =
              f32x4_mx{acc[fm][fn][4 * q], acc[fm][fn][4 * q + 1], acc[fm][fn][4 * q + 2], acc[fm][fn][4 * q + 3]};
      }
    }
  }
}

__global__ __launch_bounds__(256) void gemm1_mx_prefill(GemmArgsMX g) {
  gemm_mx_ring_body<256, 256, 2, 2, true, 2>(g);
}
__global__ __launch_bounds__(256) void gemm2_mx_prefill(GemmArgsMX g) {
  gemm_mx_ring_body<256, 256, 2, 2, false, 2>(g);
}

template <bool GATED, bool SC2>
__global__ __launch_bounds__(64 * kMxDecodeWaves) void gemm_mx_skinny(GemmArgsMX g) {
  const int L = block_tile(g);
  if (L < 0) return;
  yield_to_window(g.yield);
  TileCoord tc;
  tile_at(g, L, 32, 32 * kMxDecodeWaves, tc);
  gemm_mx_skinny_tile<GATED, SC2>(g, tc);
}

static inline int round8_mx(long long v) { return (int)((v + 7) / 8 * 8); }

hipError_t launch_ffn_mx(int regime, int gemm, const PhaseBuffers& b, const MxBuffers& mx, const MxWeights& w,
                         int e_loc, int H, int I, int max_m_tiles, YieldTo yield, hipStream_t s) {
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
  if (regime == 0) {
    g.n_tiles = gemm == 1 ? (g.N + 127) / 128 : (g.N + 255) / 256;
    const dim3 grid(round8_mx((long long)max_m_tiles * g.n_tiles));
    if (gemm == 1) gemm1_mx_prefill<<<grid, 256, 0, s>>>(g);
    else gemm2_mx_prefill<<<grid, 256, 0, s>>>(g);
  } else {
    g.n_tiles = (g.N + 32 * kMxDecodeWaves - 1) / (32 * kMxDecodeWaves);
    g.xcd_local = g.n_tiles % 8 == 0 ? 2 : 1;
    const dim3 grid(round8_mx((long long)max_m_tiles * g.n_tiles));
    const bool sc2 = g.K % 256 == 0 && ((uintptr_t)g.As | (uintptr_t)g.Bs) % 8 == 0 && g.bs_stride % 8 == 0 &&
                     ((long long)g.up_row * (g.K / 32)) % 8 == 0;
    auto go = [&](auto k) { k<<<grid, 64 * kMxDecodeWaves, 0, s>>>(g); };
    if (gemm == 1) sc2 ? go(gemm_mx_skinny<true, true>) : go(gemm_mx_skinny<true, false>);
    else sc2 ? go(gemm_mx_skinny<false, true>) : go(gemm_mx_skinny<false, false>);
  }
  return hipGetLastError();
}

int ffn_mx_bm(int regime) { return regime == 0 ? 256 : 32; }

}  // namespace moepd
