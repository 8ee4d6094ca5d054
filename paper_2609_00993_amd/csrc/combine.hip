// Weighted combine: out[t] = sum over the resident slots j of t, in slot order,
// of w[t,j] * y[row(t,j)], accumulated in float32; a token with no resident
// slot gets a zero row.  y and out are float32 for every context dtype.
// This is the receive side of the expert layer's combine (Section 2.2 /
// Section 5: DeepEP's combine returns expert outputs to their tokens)
// restricted to one GPU.
//
// A wave per token (per part of a token's row for small batches, see
// waves_per_row): lanes j < k read slot j's row and weight once, the
// resident slots become a wave-uniform bit mask, and each lane then gathers
// 16-byte vectors of y from exactly the resident rows (row ids and weights
// are read back as wave-uniform values), so y is read once per row and out
// written once per token, fully coalesced, with no per-element slot loads.
// Several resident rows are loaded before they are added, in slot order.
#include "common.h"
#include "kernels.h"

namespace moepd {

// Large batches: four 16-byte vectors per lane per pass, and up to eight
// resident rows (all of a top-8 token's) loaded together, so a pass waits
// for memory once.  y is read and out written with nontemporal accesses:
// each row of y is read once, y (2.8 GB at the 16384-token skewed batch) is
// far larger than the caches, and out lines left dirty in them would be
// written back while the next layer's dispatch runs.  At that batch the
// combine and the next permute went 667 + 297 -> 614 + 295 us alone.  Small
// batches (up to 2048 tokens, split over more waves per row): two vectors
// and two rows, plain accesses, which holds the kernel to 35 registers per
// lane, so its waves fit on a CU beside the other phase's large GEMM tiles
// (the 256-row bf16 tiles leave 52 per SIMD lane) instead of waiting for
// one of those tiles to finish (config 3, D's combine under P: 100 -> 41 us).
constexpr int kCombVec = 4, kCombGroup = 8;
constexpr int kCombVecSmall = 2, kCombGroupSmall = 2;

template <int VEC, int GROUP, bool STREAM>
__global__ __launch_bounds__(256) void combine_kernel(const u32x4* __restrict__ y, const float* __restrict__ topk_w,
                                                      const int32_t* __restrict__ row_of_slot, int T, int k, int nv,
                                                      int parts, u32x4* __restrict__ out, WindowSignal close) {
  // The layer's grouped GEMMs are done once this kernel runs: close the window.
  if (close.word && blockIdx.x == 0 && threadIdx.x == 0)
    __hip_atomic_store(close.word, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int wi = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int t = wi / parts, part = wi - t * parts;
  if (t >= T) return;  // whole wave leaves together
  const int lane = threadIdx.x & 63;
  const int r_l = lane < k ? row_of_slot[(size_t)t * k + lane] : -1;
  const float w_l = lane < k ? topk_w[(size_t)t * k + lane] : 0.f;
  const uint64_t resident = __ballot(r_l >= 0);
  u32x4* o = out + (size_t)t * nv;
  constexpr int PASS = kWave * VEC;
  for (int v0 = part * PASS; v0 < nv; v0 += parts * PASS) {
    float acc[VEC][4];
#pragma unroll
    for (int i = 0; i < VEC; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[i][e] = 0.f;
    uint64_t m = resident;
    while (m) {  // resident slots in ascending slot order, up to GROUP at a time
      int r[GROUP];
      float w[GROUP];
      int n = 0;
#pragma unroll
      for (int q = 0; q < GROUP; ++q) {
        r[q] = 0;
        w[q] = 0.f;
        if (m) {
          const int j = __builtin_ctzll(m);
          m &= m - 1;
          r[q] = __builtin_amdgcn_readlane(r_l, j);
          w[q] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w_l), j));
          n = q + 1;
        }
      }
      u32x4 a[GROUP][VEC];
#pragma unroll
      for (int q = 0; q < GROUP; ++q) {
        if (q < n) {
          const u32x4* yr = y + (size_t)r[q] * nv;
#pragma unroll
          for (int i = 0; i < VEC; ++i) {
            const int v = v0 + i * kWave + lane;
            if (v < nv) {
              if constexpr (STREAM) a[q][i] = __builtin_nontemporal_load(&yr[v]);
              else a[q][i] = yr[v];
            }
          }
        }
      }
#pragma unroll
      for (int q = 0; q < GROUP; ++q)
        if (q < n)
#pragma unroll
          for (int i = 0; i < VEC; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[i][e] += w[q] * __uint_as_float(a[q][i][e]);
    }
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      const int v = v0 + i * kWave + lane;
      if (v < nv) {
        u32x4 q;
#pragma unroll
        for (int e = 0; e < 4; ++e) q[e] = __float_as_uint(acc[i][e]);
        if constexpr (STREAM) __builtin_nontemporal_store(q, &o[v]);
        else o[v] = q;
      }
    }
  }
}

hipError_t launch_combine(const void* y, const float* topk_w, const int32_t* row_of_slot, int T, int k, int H,
                          void* out, WindowSignal close, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const int nv = H * 4 / 16;
  const bool small = T <= 2048;
  const int parts = waves_per_row(T, nv, small ? kCombVecSmall : kCombVec);
  const long long waves = (long long)T * parts;
  if (small)
    combine_kernel<kCombVecSmall, kCombGroupSmall, false><<<dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s>>>(
        (const u32x4*)y, topk_w, row_of_slot, T, k, nv, parts, (u32x4*)out, close);
  else
    combine_kernel<kCombVec, kCombGroup, true><<<dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s>>>(
        (const u32x4*)y, topk_w, row_of_slot, T, k, nv, parts, (u32x4*)out, close);
  return hipGetLastError();
}

}  // namespace moepd
