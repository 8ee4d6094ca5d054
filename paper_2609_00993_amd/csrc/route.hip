// Top-k gating: one wavefront per token.
//
// The paper routes every token to its top-k experts (Section 7.1: top-8
// routing over the routed experts) and leaves the gate to the engine.  The
// gate here is softmax over the pool, the k largest, renormalised over the k:
// w_j = exp(l_j - l_max) / sum_{i<k} exp(l_i - l_max), which is the
// renormalised softmax restricted to the selected experts.  Ties go to the
// lower expert id and -0.0 equals +0.0.
//
// Each lane holds ceil(E/64) logits as 64-bit keys (orderable logit bits in
// the high word, inverted expert id in the low word), so one wave-wide
// maximum gives the next expert of the ordering, ties included.  The k
// selections take k shuffle reductions; the selected logit of slot j ends on
// lane j, which then computes and stores its weight.
//
// After the router GEMM the kernel first forms each logit: the sum of the
// GEMM's K-split partial products in split order, plus the expert's bias if
// one is given, and stores it (the phase's logits buffer) before selecting.
#include "common.h"
#include "kernels.h"

namespace moepd {

// Monotone map of finite float32 to uint32 (larger float -> larger code),
// with -0.0 folded onto +0.0.
__device__ __forceinline__ uint32_t orderable(float v) {
  uint32_t b = __float_as_uint(v);
  if ((b & 0x7fffffffu) == 0u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float from_orderable(uint32_t o) {
  const uint32_t b = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
  return __uint_as_float(b);
}

template <int EPL>
__global__ __launch_bounds__(256) void route_kernel(const float* logits, int T, int E, int k,
                                                    int32_t* __restrict__ topk_idx, float* __restrict__ topk_w,
                                                    WindowSignal open, RouterSum sum) {
  if (open.word && blockIdx.x == 0 && threadIdx.x == 0)
    __hip_atomic_store(open.word, open.gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int lane = lane_id();
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;  // whole wave leaves together
  const float* row = logits + (size_t)t * E;

  uint64_t key[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane + i * kWave;
    float v = 0.f;
    if (e < E) {
      if (sum.out) {
        // split order, with eight loads in flight per group of adds
        const float* p = row + e;
        const size_t stride = (size_t)T * E;
        v = p[0];
        int s = 1;
        for (; s + 8 <= sum.nsplit; s += 8) {
          float a[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) a[j] = p[(s + j) * stride];
#pragma unroll
          for (int j = 0; j < 8; ++j) v += a[j];
        }
        for (; s < sum.nsplit; ++s) v += p[s * stride];
        if (sum.bias) v += sum.bias[e];
        sum.out[(size_t)t * E + e] = v;
      } else {
        v = row[e];
      }
    }
    key[i] = e < E ? ((uint64_t)orderable(v) << 32) | (uint64_t)(0xffffffffu - (uint32_t)e) : 0ull;
  }

  float my_l = 0.f, top = 0.f;
  int my_e = 0;
  for (int j = 0; j < k; ++j) {
    uint64_t best = 0ull;
#pragma unroll
    for (int i = 0; i < EPL; ++i) best = key[i] > best ? key[i] : best;
    best = wave_max_u64(best);
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (key[i] == best) key[i] = 0ull;
    const float l = from_orderable((uint32_t)(best >> 32));
    if (j == 0) top = l;
    if (lane == j) {
      my_l = l;
      my_e = (int)(0xffffffffu - (uint32_t)best);
    }
  }

  const float z = lane < k ? expf(my_l - top) : 0.f;
  float s = z;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, kWave);
  if (lane < k) {
    topk_idx[(size_t)t * k + lane] = my_e;
    topk_w[(size_t)t * k + lane] = z / s;
  }
}

hipError_t launch_route(const float* logits, int T, int E, int k, int32_t* topk_idx, float* topk_w,
                        WindowSignal open, RouterSum sum, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const dim3 grid((T + 3) / 4), block(256);
  if (E <= 64)
    route_kernel<1><<<grid, block, 0, s>>>(logits, T, E, k, topk_idx, topk_w, open, sum);
  else if (E <= 128)
    route_kernel<2><<<grid, block, 0, s>>>(logits, T, E, k, topk_idx, topk_w, open, sum);
  else if (E <= 256)
    route_kernel<4><<<grid, block, 0, s>>>(logits, T, E, k, topk_idx, topk_w, open, sum);
  else if (E <= 512)
    route_kernel<8><<<grid, block, 0, s>>>(logits, T, E, k, topk_idx, topk_w, open, sum);
  else
    route_kernel<16><<<grid, block, 0, s>>>(logits, T, E, k, topk_idx, topk_w, open, sum);
  return hipGetLastError();
}

}  // namespace moepd
