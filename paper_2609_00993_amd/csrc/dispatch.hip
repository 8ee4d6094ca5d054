// Dispatch on one GPU: the notification part (per-expert histogram and prefix
// sum, which fix the dispatch shape) and the data part (token permutation
// into expert-contiguous rows).  Section 5.2 of the paper splits normal
// dispatch exactly between these two parts.
//
// Layout contract: the rows of local expert e are [offsets[e], offsets[e+1])
// and hold its tokens in ascending token order, i.e. a stable counting sort of
// the flattened slot index t*k + j.  Every result is an integer computed
// without atomics whose outcome depends on timing: histogram cells are summed
// with LDS integer atomics (order-free), and ranks come from wave ballots
// taken in slot order, so the layout is bit-exact and reproducible.
//
// Tokens are cut into chunks of `chunk_tokens`; the count kernel writes one
// histogram cell per (expert, chunk) and its last block to arrive scans the
// cells in expert-major order, which yields the first row of every
// (expert, chunk) directly.  The place kernel then ranks the slots inside a
// chunk and adds that base.
#include "common.h"
#include "kernels.h"

namespace moepd {

__device__ __forceinline__ int local_expert(int g, int e0, int e_loc) {
  const int le = g - e0;
  return (le >= 0 && le < e_loc) ? le : -1;
}

// Block-wide exclusive scan of one int per thread (256 threads); returns the
// prefix and writes the block total to *total.
__device__ __forceinline__ int block_exclusive_scan_256(int v, int* wave_tot, int* total) {
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const int inc = wave_inclusive_scan(v);
  if (lane == kWave - 1) wave_tot[w] = inc;
  __syncthreads();
  int base = 0, all = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = wave_tot[i];
    if (i < w) base += t;
    all += t;
  }
  *total = all;
  return base + inc - v;
}

__global__ __launch_bounds__(256) void count_kernel(const int32_t* __restrict__ topk_idx, int T, int k, int e0,
                                                    int e_loc, int chunk_tokens, int nchunks, int bm,
                                                    PhaseBuffers b) {
  __shared__ int hist[kMaxLocalExperts];
  __shared__ int cells[kMaxCells];
  __shared__ int wave_tot[4];
  __shared__ int is_last;
  const int tid = threadIdx.x;
  const int c = blockIdx.x;

  for (int i = tid; i < e_loc; i += 256) hist[i] = 0;
  __syncthreads();
  const long long s0 = (long long)c * chunk_tokens * k;
  const long long t1 = min((long long)T, (long long)(c + 1) * chunk_tokens);
  const long long s1 = t1 * k;
  for (long long s = s0 + tid; s < s1; s += 256) {
    const int le = local_expert(topk_idx[s], e0, e_loc);
    if (le >= 0) atomicAdd(&hist[le], 1);
  }
  __syncthreads();
  for (int i = tid; i < e_loc; i += 256) b.chunk_counts[i * nchunks + c] = hist[i];

  // Publish the cells, then count arrivals; the last block does the scan.
  __threadfence();
  __syncthreads();
  if (tid == 0) is_last = (atomicAdd(b.done, 1u) == (unsigned)(nchunks - 1));
  __syncthreads();
  if (!is_last) return;
  __threadfence();

  const int n = e_loc * nchunks;  // <= kMaxCells (host guarantees)
  for (int i = tid; i < n; i += 256) cells[i] = __atomic_load_n(&b.chunk_counts[i], __ATOMIC_RELAXED);
  __syncthreads();
  // each thread owns a contiguous segment of cells
  const int seg = (n + 255) / 256;
  const int lo = min(n, tid * seg), hi = min(n, lo + seg);
  int sum = 0;
  for (int i = lo; i < hi; ++i) sum += cells[i];
  int total;
  int run = block_exclusive_scan_256(sum, wave_tot, &total);
  for (int i = lo; i < hi; ++i) {
    const int v = cells[i];
    b.chunk_base[i] = run;
    cells[i] = run;  // exclusive prefix, expert-major
    run += v;
  }
  __syncthreads();
  // offsets[e] = first row of (e, chunk 0); counts from consecutive offsets
  for (int e = tid; e < e_loc; e += 256) {
    const int off = cells[e * nchunks];
    const int nxt = (e + 1 < e_loc) ? cells[(e + 1) * nchunks] : total;
    b.offsets[e] = off;
    b.counts[e] = nxt - off;
    hist[e] = (nxt - off + bm - 1) / bm;  // m-tiles of expert e
  }
  if (tid == 0) b.offsets[e_loc] = total;
  __syncthreads();
  if (tid == 0) {
    int acc = 0;
    for (int e = 0; e < e_loc; ++e) {
      b.tile_base[e] = acc;
      acc += hist[e];
    }
    b.tile_base[e_loc] = acc;
    __atomic_store_n(b.done, 0u, __ATOMIC_RELAXED);  // ready for the next call
  }
}

__global__ __launch_bounds__(256) void place_kernel(const int32_t* __restrict__ topk_idx, int T, int k, int e0,
                                                    int e_loc, int chunk_tokens, int nchunks, int nbits,
                                                    PhaseBuffers b) {
  __shared__ int run[kMaxLocalExperts + 1];
  __shared__ int wcnt[4][kMaxLocalExperts + 1];
  const int tid = threadIdx.x, w = tid >> 6;
  const int c = blockIdx.x;
  for (int i = tid; i <= e_loc; i += 256) {
    run[i] = 0;
    wcnt[0][i] = wcnt[1][i] = wcnt[2][i] = wcnt[3][i] = 0;
  }
  __syncthreads();
  const long long s0 = (long long)c * chunk_tokens * k;
  const long long s1 = min((long long)T, (long long)(c + 1) * chunk_tokens) * k;
  const uint64_t lt = lanemask_lt();

  for (long long base = s0; base < s1; base += 256) {
    const long long s = base + tid;
    const bool valid = s < s1;
    const int le = valid ? local_expert(topk_idx[s], e0, e_loc) : -1;
    const int cat = le + 1;  // 0 = dropped or past the chunk
    // lanes of this wave with the same category, via one ballot per bit
    uint64_t match = ~0ull;
    for (int bit = 0; bit < nbits; ++bit) {
      const bool on = (cat >> bit) & 1;
      const uint64_t bal = __ballot(on);
      match &= on ? bal : ~bal;
    }
    const int rank = __popcll(match & lt);
    if (rank == 0 && cat > 0) wcnt[w][cat] = __popcll(match);
    __syncthreads();
    if (valid) {
      if (le >= 0) {
        int pre = run[cat];
        for (int v = 0; v < w; ++v) pre += wcnt[v][cat];
        const int row = b.chunk_base[le * nchunks + c] + pre + rank;
        b.row_of_slot[s] = row;
        b.token_of_row[row] = (int)(s / k);
      } else {
        b.row_of_slot[s] = -1;
      }
    }
    __syncthreads();
    for (int i = tid; i <= e_loc; i += 256) {
      run[i] += wcnt[0][i] + wcnt[1][i] + wcnt[2][i] + wcnt[3][i];
      wcnt[0][i] = wcnt[1][i] = wcnt[2][i] = wcnt[3][i] = 0;
    }
    __syncthreads();
  }
}

// Token-major scatter: each 16-byte vector of x[t] is read once and written to
// every row that t occupies, so HBM sees (tokens + rows) x row bytes.
constexpr int kPermItems = 4;

__global__ __launch_bounds__(256) void permute_kernel(const uint8_t* __restrict__ x, int T, int k, int nv,
                                                      int tokens_per_block, const int32_t* __restrict__ row_of_slot,
                                                      uint8_t* __restrict__ x_perm) {
  const int t_begin = blockIdx.x * tokens_per_block;
  const int t_end = min(T, t_begin + tokens_per_block);
  const int items = (t_end - t_begin) * nv;
  for (int base = 0; base < items; base += 256 * kPermItems) {
    u32x4 v[kPermItems];
    int tt[kPermItems], vi[kPermItems];
#pragma unroll
    for (int i = 0; i < kPermItems; ++i) {
      const int it = base + i * 256 + (int)threadIdx.x;
      tt[i] = -1;
      if (it < items) {
        const int tl = it / nv;
        tt[i] = t_begin + tl;
        vi[i] = it - tl * nv;
        v[i] = load16(x + ((size_t)tt[i] * nv + vi[i]) * 16);
      }
    }
#pragma unroll
    for (int i = 0; i < kPermItems; ++i) {
      if (tt[i] < 0) continue;
      const int32_t* rs = row_of_slot + (size_t)tt[i] * k;
      for (int j = 0; j < k; ++j) {
        const int r = rs[j];
        if (r >= 0) store16(x_perm + ((size_t)r * nv + vi[i]) * 16, v[i]);
      }
    }
  }
}

hipError_t launch_count(const int32_t* topk_idx, int T, int k, int e0, int e_loc, int chunk_tokens, int nchunks,
                        int bm, const PhaseBuffers& b, hipStream_t s) {
  count_kernel<<<dim3(nchunks), dim3(256), 0, s>>>(topk_idx, T, k, e0, e_loc, chunk_tokens, nchunks, bm, b);
  return hipGetLastError();
}

hipError_t launch_place(const int32_t* topk_idx, int T, int k, int e0, int e_loc, int chunk_tokens, int nchunks,
                        const PhaseBuffers& b, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  int nbits = 0;
  while ((1 << nbits) <= e_loc) ++nbits;  // categories 0..e_loc
  place_kernel<<<dim3(nchunks), dim3(256), 0, s>>>(topk_idx, T, k, e0, e_loc, chunk_tokens, nchunks, nbits, b);
  return hipGetLastError();
}

hipError_t launch_permute(const void* x, int T, int k, int row_bytes, const int32_t* row_of_slot, void* x_perm,
                          hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const int nv = row_bytes / 16;
  int tpb = 1024 / nv;
  if (tpb < 1) tpb = 1;
  const int grid = (T + tpb - 1) / tpb;
  permute_kernel<<<dim3(grid), dim3(256), 0, s>>>((const uint8_t*)x, T, k, nv, tpb, row_of_slot,
                                                  (uint8_t*)x_perm);
  return hipGetLastError();
}

}  // namespace moepd
