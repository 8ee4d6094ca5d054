// Weighted combine: out[t] = sum over the resident slots j of t, in slot order,
// of w[t,j] * y[row(t,j)], accumulated in float32; a token with no resident
// slot gets a zero row.  y and out are float32 for every context dtype.  This is the receive side of the expert layer's
// combine (Section 2.2 / Section 5: DeepEP's combine returns expert outputs
// to their tokens) restricted to one GPU.
//
// Token-major gather: every 16-byte vector of out[t] is produced by one lane
// from the matching vectors of t's rows, so y is read once per row and out is
// written once per token, both fully coalesced.
#include "common.h"
#include "kernels.h"

namespace moepd {

constexpr int kCombItems = 2;

__global__ __launch_bounds__(256) void combine_kernel(const uint8_t* __restrict__ y, const float* __restrict__ topk_w,
                                                      const int32_t* __restrict__ row_of_slot, int T, int k, int nv,
                                                      int tokens_per_block, uint8_t* __restrict__ out) {
  const int t_begin = blockIdx.x * tokens_per_block;
  const int t_end = min(T, t_begin + tokens_per_block);
  const int items = (t_end - t_begin) * nv;
  for (int base = 0; base < items; base += 256 * kCombItems) {
#pragma unroll
    for (int i = 0; i < kCombItems; ++i) {
      const int it = base + i * 256 + (int)threadIdx.x;
      if (it >= items) continue;
      const int tl = it / nv;
      const int t = t_begin + tl;
      const int vi = it - tl * nv;
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
      const int32_t* rs = row_of_slot + (size_t)t * k;
      const float* ws = topk_w + (size_t)t * k;
      for (int j = 0; j < k; ++j) {
        const int r = rs[j];
        if (r < 0) continue;
        const float wt = ws[j];
        const u32x4 a = load16(y + ((size_t)r * nv + vi) * 16);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] += wt * __uint_as_float(a[e]);
      }
      u32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = __float_as_uint(acc[e]);
      store16(out + ((size_t)t * nv + vi) * 16, o);
    }
  }
}

hipError_t launch_combine(const void* y, const float* topk_w, const int32_t* row_of_slot, int T, int k, int H,
                          void* out, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const int nv = H * 4 / 16;
  int tpb = 512 / nv;
  if (tpb < 1) tpb = 1;
  const int grid = (T + tpb - 1) / tpb;
  combine_kernel<<<dim3(grid), dim3(256), 0, s>>>((const uint8_t*)y, topk_w, row_of_slot, T, k, nv, tpb,
                                                  (uint8_t*)out);
  return hipGetLastError();
}

}  // namespace moepd
