// Engine clock probe: the shader clock over a spin timed by the 100 MHz
// reference counter, so results can be read against clock-derived peaks.
#include <stdint.h>

#include "moepd.h"
#include "common.h"

namespace moepd {

__global__ __launch_bounds__(64) void clock_probe_kernel(uint64_t ref_ticks, uint64_t* out) {
  const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
  const uint64_t c0 = __builtin_amdgcn_s_memtime();
  uint64_t r = r0;
  // the reference counter always advances, so the spin ends
  while (r - r0 < ref_ticks) {
    __builtin_amdgcn_s_sleep(2);
    r = __builtin_amdgcn_s_memrealtime();
  }
  const uint64_t c1 = __builtin_amdgcn_s_memtime();
  if (threadIdx.x == 0) {
    out[0] = c1 - c0;
    out[1] = r - r0;
  }
}

}  // namespace moepd

extern "C" int moe_clock_probe(hipStream_t stream, int32_t spin_us, uint64_t* out_dev) {
  if (!stream || !out_dev || spin_us < 1 || spin_us > 100000) return MOE_ERR_INVALID_ARG;
  moepd::clock_probe_kernel<<<dim3(1), dim3(64), 0, stream>>>((uint64_t)spin_us * 100u, out_dev);
  return hipGetLastError() == hipSuccess ? MOE_OK : MOE_ERR_HIP;
}
