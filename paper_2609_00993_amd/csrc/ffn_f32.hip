// Grouped expert FFN in float32 (contexts created with MOE_DTYPE_F32).
//
// Same contraction and device-side tile schedule as the bf16 path (see
// ffn_bf16.hip): GEMM1 h = silu(x_perm W1^T) * (x_perm W3^T) with the SwiGLU
// in the epilogue, GEMM2 y = h W2^T, rows of expert e = [offsets[e],
// offsets[e+1]).  Products and sums are float32 FMAs on the vector ALUs; the
// float32 layer is small (it serves as the exact-arithmetic check of the
// layer), so a plain 64x64 LDS tile with 4x4 outputs per thread suffices.
#include "common.h"
#include "kernels.h"

namespace moepd {

struct GemmArgsF {
  const float* A;
  const float* B;
  float* C;
  const int32_t* offsets;
  const int32_t* tile_base;
  long long b_stride;
  int e_loc, N, K, n_tiles, up_row;
};

// Tile of this workgroup (same schedule as the bf16 path); tile_base and
// offsets are copied to LDS first so the search costs one memory latency.
__device__ __forceinline__ bool tile_lookup_f(const GemmArgsF& g, int bm, int bn, int& e, int& m0, int& m_end,
                                              int& n0) {
  __shared__ int s_tb[kMaxLocalExperts + 1];
  __shared__ int s_off[kMaxLocalExperts + 1];
  for (int i = threadIdx.x; i <= g.e_loc; i += blockDim.x) {
    s_tb[i] = g.tile_base[i];
    s_off[i] = g.offsets[i];
  }
  __syncthreads();
  const int total = s_tb[g.e_loc] * g.n_tiles;
  const int per_xcd = (total + 7) >> 3;
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  if (slot >= per_xcd) return false;
  const int L = xcd * per_xcd + slot;
  if (L >= total) return false;
  int lo = 0, hi = g.e_loc - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_tb[mid] * g.n_tiles <= L) lo = mid;
    else hi = mid - 1;
  }
  e = lo;
  const int mt_e = s_tb[e + 1] - s_tb[e];
  const int local = L - s_tb[e] * g.n_tiles;
  const int nt = local / mt_e, mt = local - nt * mt_e;
  m0 = s_off[e] + mt * bm;
  m_end = s_off[e + 1];
  n0 = nt * bn;
  return true;
}

template <bool GATED>
__global__ __launch_bounds__(256) void gemm_f32(GemmArgsF g) {
  constexpr int BM = 64, BN = 64, BK = 16;
  constexpr int NB = GATED ? 2 : 1;
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[NB][BK][BN + 4];
  int e, m0, m_end, n0;
  if (!tile_lookup_f(g, BM, BN, e, m0, m_end, n0)) return;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const float* Be = g.B + (size_t)e * g.b_stride;

  float acc[NB][4][4];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[nb][i][j] = 0.f;

  for (int k0 = 0; k0 < g.K; k0 += BK) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int q = tid + i * 256, r = q >> 4, kk = q & 15;
      const int row = min(m0 + r, m_end - 1);
      As[kk][r] = g.A[(size_t)row * g.K + k0 + kk];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int brow = nb * g.up_row + min(n0 + r, g.N - 1);
        Bs[nb][kk][r] = Be[(size_t)brow * g.K + k0 + kk];
      }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float a[4], bv[NB][4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int j = 0; j < 4; ++j) bv[nb][j] = Bs[nb][kk][tx * 4 + j];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[nb][i][j] = fmaf(a[i], bv[nb][j], acc[nb][i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= m_end) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx * 4 + j;
      if (col >= g.N) continue;
      float v = acc[0][i][j];
      if (GATED) {
        const float gt = acc[0][i][j];
        v = gt / (1.f + expf(-gt)) * acc[NB - 1][i][j];
      }
      g.C[(size_t)row * g.N + col] = v;
    }
  }
}

int ffn_f32_bm() { return 64; }

hipError_t launch_ffn_f32(int gemm, const PhaseBuffers& b, const void* w_gu, const void* w_dn, int e_loc, int H,
                          int I, int max_m_tiles, hipStream_t s) {
  GemmArgsF g;
  g.offsets = b.offsets;
  g.tile_base = b.tile_base;
  g.e_loc = e_loc;
  if (gemm == 1) {
    g.A = (const float*)b.x_perm;
    g.B = (const float*)w_gu;
    g.C = (float*)b.h;
    g.b_stride = 2LL * I * H;
    g.N = I;
    g.K = H;
    g.up_row = I;
  } else {
    g.A = (const float*)b.h;
    g.B = (const float*)w_dn;
    g.C = b.y;
    g.b_stride = (long long)H * I;
    g.N = H;
    g.K = I;
    g.up_row = 0;
  }
  g.n_tiles = (g.N + 63) / 64;
  const long long blocks = ((long long)max_m_tiles * g.n_tiles + 7) / 8 * 8;
  if (gemm == 1)
    gemm_f32<true><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(g);
  else
    gemm_f32<false><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(g);
  return hipGetLastError();
}

// Router GEMM of float32 contexts: one wave per token, lane l computes the
// logits of experts l, l + 64, ... as a sequential float32 FMA chain over h
// (x[t][h] is the same address for every lane of the wave).
__global__ __launch_bounds__(256) void router_f32(const float* __restrict__ x, const float* __restrict__ w, int T,
                                                  int E, int H, float* __restrict__ out) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const int lane = threadIdx.x & 63;
  const float* xr = x + (size_t)t * H;
  for (int e = lane; e < E; e += 64) {
    const float* wr = w + (size_t)e * H;
    float acc = 0.f;
    for (int h = 0; h < H; ++h) acc = fmaf(xr[h], wr[h], acc);
    out[(size_t)t * E + e] = acc;
  }
}

hipError_t launch_router_f32(const float* x, const float* w, int T, int E, int H, float* out, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  router_f32<<<dim3((T + 3) / 4), dim3(256), 0, s>>>(x, w, T, E, H, out);
  return hipGetLastError();
}

}  // namespace moepd
