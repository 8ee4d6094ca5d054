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
// Tokens are cut into chunks of `chunk_tokens` (a small batch is one chunk,
// which the place kernel counts itself).  The count kernel writes one
// histogram cell per (expert, chunk).  The place kernel (the next launch, so
// every cell is visible without device-scope fences) scans the cells in
// expert-major order in LDS, which yields the first row of every (expert,
// chunk) directly; its block 0 also publishes counts, offsets and the m-tile
// prefix for the FFN.  Each block then ranks the slots of its own chunk.
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

// Slot (or cell) loads each thread keeps in flight: the layout kernels are
// latency-bound, so a loop that loads one value and then waits on it would
// pay a full memory round trip per 256 slots.
constexpr int kLoadBatch = 8;
static_assert(kOneChunkSlots <= kLoadBatch * 256, "a one-chunk batch is loaded in one go");

// Category of slot s of [0, s1): its local expert + 1, or 0 (dropped or past
// the end), for the kLoadBatch slots sb + 256 j + threadIdx.x.
__device__ __forceinline__ void load_cats(const int32_t* __restrict__ topk_idx, long long sb, long long s1, int e0,
                                          int e_loc, int (&cat)[kLoadBatch]) {
#pragma unroll
  for (int j = 0; j < kLoadBatch; ++j) {
    const long long s = sb + (long long)j * 256 + threadIdx.x;
    cat[j] = s < s1 ? local_expert(topk_idx[s], e0, e_loc) + 1 : 0;
  }
}

__global__ __launch_bounds__(256) void count_kernel(const int32_t* __restrict__ topk_idx, int T, int k, int e0,
                                                    int e_loc, int chunk_tokens, int nchunks,
                                                    int32_t* __restrict__ cells) {
  __shared__ int hist[kMaxLocalExperts];
  const int tid = threadIdx.x;
  const int c = blockIdx.x;
  for (int i = tid; i < e_loc; i += 256) hist[i] = 0;
  __syncthreads();
  const long long s0 = (long long)c * chunk_tokens * k;
  const long long s1 = min((long long)T, (long long)(c + 1) * chunk_tokens) * k;
  for (long long sb = s0; sb < s1; sb += kLoadBatch * 256) {
    int cat[kLoadBatch];
    load_cats(topk_idx, sb, s1, e0, e_loc, cat);
#pragma unroll
    for (int j = 0; j < kLoadBatch; ++j)
      if (cat[j] > 0) atomicAdd(&hist[cat[j] - 1], 1);
  }
  __syncthreads();
  for (int i = tid; i < e_loc; i += 256) cells[i * nchunks + c] = hist[i];
}

// LDS word of histogram cell i (one pad word after every 32), and the words
// that n cells take.
__device__ __host__ __forceinline__ int cix(int i) { return i + (i >> 5); }
__device__ __host__ __forceinline__ int cell_words(int n) { return n + (n >> 5) + 1; }

__global__ __launch_bounds__(256) void place_kernel(const int32_t* __restrict__ topk_idx, int T, int k, int e0,
                                                    int e_loc, int chunk_tokens, int nchunks, int nbits, int bm,
                                                    PhaseBuffers b) {
  // LDS: the cells (sized at launch to e_loc * nchunks, so a small batch
  // needs only a few KB and can share a CU with a running prefill GEMM),
  // then per-expert bases, running counts and per-wave counts.
  extern __shared__ int lds_dyn[];
  // The cells sit in LDS with one pad word after every 32 (index cix(i)):
  // the scan's per-thread runs of consecutive cells and the per-expert reads
  // at stride nchunks would otherwise fall on one or two of the 64 banks.
  int* cells = lds_dyn;
  int* base = cells + cell_words(e_loc * nchunks);
  int* run = base + e_loc;
  const int ws = e_loc + 1;    // row stride of the per-wave counts
  int* wcnt = run + e_loc + 1;  // [4][e_loc + 1]
  __shared__ int wave_tot[4];
  const int tid = threadIdx.x, w = tid >> 6;
  const int c = blockIdx.x;
  const long long s0 = (long long)c * chunk_tokens * k;
  const long long s1 = min((long long)T, (long long)(c + 1) * chunk_tokens) * k;

  // categories of this chunk's first kLoadBatch * 256 slots (all of them for
  // a one-chunk batch), loaded once for the count and the ranks
  int cat0[kLoadBatch];
  load_cats(topk_idx, s0, s1, e0, e_loc, cat0);

  // exclusive scan of all (expert, chunk) cells, expert-major
  const int n = e_loc * nchunks;  // <= kMaxCells (host guarantees)
  if (nchunks == 1) {
    // one chunk: count its slots here (LDS integer atomics, order-free)
    for (int i = tid; i < n; i += 256) cells[cix(i)] = 0;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kLoadBatch; ++j)
      if (cat0[j] > 0) atomicAdd(&cells[cix(cat0[j] - 1)], 1);
    for (long long sb = s0 + kLoadBatch * 256; sb < s1; sb += kLoadBatch * 256) {
      int cat[kLoadBatch];
      load_cats(topk_idx, sb, s1, e0, e_loc, cat);
#pragma unroll
      for (int j = 0; j < kLoadBatch; ++j)
        if (cat[j] > 0) atomicAdd(&cells[cix(cat[j] - 1)], 1);
    }
  } else {
    // every cell in one round of loads (the count kernel's blocks wrote them
    // through other XCDs' caches, so each load is a trip past this L2)
    constexpr int kCellLoads = kMaxCells / 256;
    int v[kCellLoads];
#pragma unroll
    for (int j = 0; j < kCellLoads; ++j) {
      const int i = j * 256 + tid;
      v[j] = i < n ? b.chunk_counts[i] : 0;
    }
#pragma unroll
    for (int j = 0; j < kCellLoads; ++j) {
      const int i = j * 256 + tid;
      if (i < n) cells[cix(i)] = v[j];
    }
  }
  __syncthreads();
  const int seg = (n + 255) / 256;
  const int lo = min(n, tid * seg), hi = min(n, lo + seg);
  int sum = 0;
  for (int i = lo; i < hi; ++i) sum += cells[cix(i)];
  int total;
  int acc = block_exclusive_scan_256(sum, wave_tot, &total);
  __syncthreads();  // every thread has read wave_tot; cells are rewritten below
  for (int i = lo; i < hi; ++i) {
    const int v = cells[cix(i)];
    cells[cix(i)] = acc;
    acc += v;
  }
  __syncthreads();
  // e_loc <= kMaxLocalExperts = 256: thread e owns expert e below
  if (tid < e_loc) base[tid] = cells[cix(tid * nchunks + c)];
  if (c == 0) {
    // publish the dispatch shape: counts, offsets, and the m-tile prefix
    // (a block scan of the per-expert m-tile counts)
    int mt = 0;
    if (tid < e_loc) {
      const int off = cells[cix(tid * nchunks)];
      const int nxt = (tid + 1 < e_loc) ? cells[cix((tid + 1) * nchunks)] : total;
      b.offsets[tid] = off;
      b.counts[tid] = nxt - off;
      mt = (nxt - off + bm - 1) / bm;
    }
    int mt_total;
    const int tb = block_exclusive_scan_256(mt, wave_tot, &mt_total);
    if (tid < e_loc) b.tile_base[tid] = tb;
    if (tid == 0) {
      b.offsets[e_loc] = total;
      b.tile_base[e_loc] = mt_total;
    }
  }
  for (int i = tid; i <= e_loc; i += 256) {
    run[i] = 0;
    wcnt[i] = wcnt[ws + i] = wcnt[2 * ws + i] = wcnt[3 * ws + i] = 0;
  }
  __syncthreads();

  // stable ranks of this chunk's slots, 256 slots per round, in slot order
  const uint64_t lt = lanemask_lt();
  for (long long sb0 = s0; sb0 < s1; sb0 += kLoadBatch * 256) {
    int cat_r[kLoadBatch];
    if (sb0 == s0) {
#pragma unroll
      for (int j = 0; j < kLoadBatch; ++j) cat_r[j] = cat0[j];
    } else {
      load_cats(topk_idx, sb0, s1, e0, e_loc, cat_r);
    }
#pragma unroll
    for (int j = 0; j < kLoadBatch; ++j) {
      const long long sb = sb0 + (long long)j * 256;
      if (sb >= s1) break;  // block-uniform
      const long long s = sb + tid;
      const bool valid = s < s1;
      const int cat = cat_r[j];  // 0 = dropped or past the chunk
      const int le = cat - 1;
      // lanes of this wave with the same category, via one ballot per bit
      uint64_t match = ~0ull;
      for (int bit = 0; bit < nbits; ++bit) {
        const bool on = (cat >> bit) & 1;
        const uint64_t bal = __ballot(on);
        match &= on ? bal : ~bal;
      }
      const int rank = __popcll(match & lt);
      if (rank == 0 && cat > 0) wcnt[w * ws + cat] = __popcll(match);
      __syncthreads();
      if (valid) {
        if (le >= 0) {
          int pre = run[cat];
          for (int v = 0; v < w; ++v) pre += wcnt[v * ws + cat];
          const int row = base[le] + pre + rank;
          b.row_of_slot[s] = row;
          b.token_of_row[row] = (int)(s / k);
        } else {
          b.row_of_slot[s] = -1;
        }
      }
      __syncthreads();
      for (int i = tid; i <= e_loc; i += 256) {
        run[i] += wcnt[i] + wcnt[ws + i] + wcnt[2 * ws + i] + wcnt[3 * ws + i];
        wcnt[i] = wcnt[ws + i] = wcnt[2 * ws + i] = wcnt[3 * ws + i] = 0;
      }
      __syncthreads();
    }
  }
}

// Token-major scatter, one wave per token (per part of its row for small
// batches, see waves_per_row): lanes j < k read slot j's row, the
// resident slots become a wave-uniform bit mask, and each 16-byte vector of
// x[t] is read once and written to every row t occupies (row ids read back
// as wave-uniform values).  Tokens with no resident slot are not read, so HBM
// sees (tokens with a resident slot + rows) x row bytes.
constexpr int kPermVec = 4;  // 16-byte vectors per lane per pass

__global__ __launch_bounds__(256) void permute_kernel(const u32x4* __restrict__ x, int T, int k, int nv,
                                                      int parts, const int32_t* __restrict__ row_of_slot,
                                                      u32x4* __restrict__ x_perm) {
  const int wi = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int t = wi / parts, part = wi - t * parts;
  if (t >= T) return;  // whole wave leaves together
  const int lane = threadIdx.x & 63;
  const int r_l = lane < k ? row_of_slot[(size_t)t * k + lane] : -1;
  const uint64_t resident = __ballot(r_l >= 0);
  if (!resident) return;
  const u32x4* xt = x + (size_t)t * nv;
  for (int v0 = part * kWave * kPermVec; v0 < nv; v0 += parts * kWave * kPermVec) {
    u32x4 a[kPermVec];
#pragma unroll
    for (int i = 0; i < kPermVec; ++i) {
      const int v = v0 + i * kWave + lane;
      if (v < nv) a[i] = xt[v];
    }
    uint64_t m = resident;
    while (m) {
      const int j = __builtin_ctzll(m);
      m &= m - 1;
      u32x4* dst = x_perm + (size_t)__builtin_amdgcn_readlane(r_l, j) * nv;
#pragma unroll
      for (int i = 0; i < kPermVec; ++i) {
        const int v = v0 + i * kWave + lane;
        if (v < nv) dst[v] = a[i];
      }
    }
  }
}

hipError_t launch_count(const int32_t* topk_idx, int T, int k, int e0, int e_loc, int chunk_tokens, int nchunks,
                        const PhaseBuffers& b, hipStream_t s) {
  count_kernel<<<dim3(nchunks), dim3(256), 0, s>>>(topk_idx, T, k, e0, e_loc, chunk_tokens, nchunks,
                                                   b.chunk_counts);
  return hipGetLastError();
}

hipError_t launch_place(const int32_t* topk_idx, int T, int k, int e0, int e_loc, int chunk_tokens, int nchunks,
                        int bm, const PhaseBuffers& b, hipStream_t s) {
  int nbits = 0;
  while ((1 << nbits) <= e_loc) ++nbits;  // categories 0..e_loc
  const size_t lds = sizeof(int) * ((size_t)cell_words(e_loc * nchunks) + e_loc + 5 * (size_t)(e_loc + 1));
  place_kernel<<<dim3(nchunks), dim3(256), lds, s>>>(topk_idx, T, k, e0, e_loc, chunk_tokens, nchunks, nbits, bm, b);
  return hipGetLastError();
}

hipError_t launch_permute(const void* x, int T, int k, int row_bytes, const int32_t* row_of_slot, void* x_perm,
                          hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const int nv = row_bytes / 16;
  const int parts = waves_per_row(T, nv, kPermVec);
  const long long waves = (long long)T * parts;
  permute_kernel<<<dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s>>>((const u32x4*)x, T, k, nv, parts,
                                                                          row_of_slot, (u32x4*)x_perm);
  return hipGetLastError();
}

}  // namespace moepd
