// The dispatch layout (the notification half of dispatch, Section 5.2) for
// callers that cannot allocate device memory: code under graph capture,
// tight serving loops, harnesses that forbid allocation.  The caller passes
// the routing indices and the four layout outputs; the kernels are those of
// moe_dispatch_layout, and their scratch (the per-chunk histogram cells and
// the m-tile prefix) lives in a fixed device array of this file instead of a
// context's phase allocation.
//
// Each device holds its own copy of the array until the process ends.  Its
// device address is looked up once per device (hipGetSymbolAddress, with that
// device current) on the entry point's first call there, and only that address
// reaches the kernels.  Every call on a device shares the array: calls that
// overlap on one device (two streams, or two host threads) race on it.  No
// cell has to start at zero: the count kernel writes every cell the place
// kernel reads, and a batch of one chunk is counted in LDS.
#include <mutex>

#include "kernels.h"
#include "moepd.h"

using namespace moepd;

// The cells (at most kMaxCells, the chunking's bound) and the m-tile prefix
// (at most kMaxLocalExperts + 1 entries): 33,796 bytes.  In host code the
// name stands for the array, not for its device address: only the address
// looked up by scratch_on reaches a kernel.
constexpr int kScratchWords = kMaxCells + kMaxLocalExperts + 1;
static __device__ __align__(256) int32_t scratch[kScratchWords];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
int32_t* g_scratch[kMaxDevices] = {};  // device address of `scratch` on each device

// The device address of this device's scratch array (looked up once).
int scratch_on(int dev, int32_t** out) {
  if (dev < 0 || dev >= kMaxDevices) return MOE_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return MOE_ERR_HIP;
    }
    g_scratch[dev] = static_cast<int32_t*>(p);
  }
  *out = g_scratch[dev];
  return MOE_OK;
}

// m-tile height handed to the place kernel: its m-tile prefix only feeds the
// grouped GEMMs, which this entry point does not launch.
constexpr int kPrefixTileRows = 32;

}  // namespace

extern "C" int moe_dispatch_layout_noalloc(const int32_t* topk_idx, int32_t T, int32_t top_k, int32_t expert_begin,
                                           int32_t num_local_experts, int32_t* counts, int32_t* offsets,
                                           int32_t* row_of_slot, int32_t* token_of_row, hipStream_t stream) {
  if (T < 0 || top_k < 1 || top_k > kMaxTopK || expert_begin < 0 || num_local_experts < 1 ||
      num_local_experts > kMaxLocalExperts || !counts || !offsets || !stream)
    return MOE_ERR_INVALID_ARG;
  if (T > 0 && (!topk_idx || !row_of_slot || !token_of_row)) return MOE_ERR_INVALID_ARG;
  if (T > MOE_NOALLOC_MAX_TOKENS) return MOE_ERR_CAPACITY;
  int chunk_tokens = 1, nchunks = 1;
  dispatch_chunking(T, top_k, num_local_experts, &chunk_tokens, &nchunks);
  if ((long long)nchunks * num_local_experts > kMaxCells) return MOE_ERR_CAPACITY;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MOE_ERR_HIP;
  int32_t* sc = nullptr;
  int st = scratch_on(dev, &sc);
  if (st) return st;
  PhaseBuffers b{};
  b.counts = counts;
  b.offsets = offsets;
  b.row_of_slot = row_of_slot;
  b.token_of_row = token_of_row;
  b.chunk_counts = sc;
  b.tile_base = sc + kMaxCells;
  if (nchunks > 1 &&
      launch_count(topk_idx, T, top_k, expert_begin, num_local_experts, chunk_tokens, nchunks, b, stream) != hipSuccess)
    return MOE_ERR_HIP;
  if (launch_place(topk_idx, T, top_k, expert_begin, num_local_experts, chunk_tokens, nchunks, kPrefixTileRows, b,
                   stream) != hipSuccess)
    return MOE_ERR_HIP;
  return MOE_OK;
}
