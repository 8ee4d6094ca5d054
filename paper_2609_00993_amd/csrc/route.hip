// Top-k gating: one wavefront per token.
//
// The paper routes every token to its top-k experts (Section 7.1: top-8
// routing over the routed experts) and leaves the gate to the engine.  The
// gate here is softmax over the pool, the k largest, renormalised over the k:
// w_j = exp(l_j - l_max) / sum_{i<k} exp(l_i - l_max), which is the
// renormalised softmax restricted to the selected experts.  Ties go to the
// lower expert id and -0.0 equals +0.0.
//
// Each lane holds ceil(E/64) logits as 32-bit orderable keys (larger logit,
// larger key; expert e = lane + 64 i sits in the lane's slot i).  Selection
// j takes the wave maximum M of the remaining keys, then the wave minimum of
// the expert ids whose key is M (ties go to the lower id), and retires that
// expert's key.  Both reductions are 32-bit DPP maxima/minima, full-rate
// instructions, where one 64-bit (key, id) reduction would take compare and
// select pairs per step.  The selected logit of slot j ends on lane j, which
// then computes and stores its weight.
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

  uint32_t key[EPL];  // 0 = no expert / taken (every finite logit's key is larger)
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
    key[i] = e < E ? orderable(v) : 0u;
  }

  float my_l = 0.f, top = 0.f;
  int my_e = 0;
  for (int j = 0; j < k; ++j) {
    uint32_t m = 0u;
#pragma unroll
    for (int i = 0; i < EPL; ++i) m = key[i] > m ? key[i] : m;
    const uint32_t best = wave_max_u32(m);
    // the lowest expert id holding `best` (slot order is id order)
    uint32_t cand = 0xffffffffu;
#pragma unroll
    for (int i = EPL - 1; i >= 0; --i)
      if (key[i] == best) cand = (uint32_t)(lane + i * kWave);
    const uint32_t win = wave_min_u32(cand);
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if ((uint32_t)(lane + i * kWave) == win) key[i] = 0u;
    const float l = from_orderable(best);
    if (j == 0) top = l;
    if (lane == j) {
      my_l = l;
      my_e = (int)win;
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
