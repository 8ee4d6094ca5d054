// Tile scheduling shared by the grouped GEMMs (bf16 and MX FP8): logical
// tile ids, their (expert, row block, column block) coordinates, and the
// XCD-aware mapping of workgroups to tiles.  The mapping itself is plain
// arithmetic, compiled for the host too, where a test checks it.  G is a GEMM argument struct
// with offsets, tile_base, e_loc, n_tiles, n_group and xcd_local (and the
// dense_* fields for the dense mode).
#pragma once

#include <hip/hip_runtime.h>

#include "kernels.h"

namespace moepd {

struct TileCoord {
  int e, m0, m_end, n0;
  int split;  // K split of a dense tile (0 otherwise)
};

// Tile of a dense GEMM: splits outermost, then m-tiles, n-tile fastest (the
// n-tiles of one row block run side by side and share its activation rows).
template <class G>
__host__ __device__ __forceinline__ void dense_tile_at(const G& g, int L, int bm, int bn, TileCoord& tc) {
  const int per_split = g.dense_total / g.dense_splits;
  const int s = L / per_split, r = L - s * per_split;
  const int mt = r / g.n_tiles;
  tc.e = 0;
  tc.m0 = mt * bm;
  tc.m_end = g.dense_rows;
  tc.n0 = (r - mt * g.n_tiles) * bn;
  tc.split = s;
}

// Coordinates of logical tile L.  Tiles run expert-major.  Within an expert
// (mt m-tiles x n_tiles n-tiles), optionally cut into super-rows of m_super
// m-tiles taken one after another, the n-tiles are cut into blocks of
// n_group; block by block, the tiles go m-tile by m-tile, n-tile fastest.  So
// consecutive tiles (which one XCD runs side by side, see block_tile) share
// an activation row block across n_group n-tiles and a weight n-tile across
// the m-tiles running together.  n_group = n_tiles is plain m-major order.
// With XCD-local tiles an expert's rows are shared evenly among its m-tiles
// (tile_base counts ceil(rows / bm) of them, so none holds more than bm rows
// and none is empty): the m-tiles that stream one weight panel on one XCD
// then move at one pace and keep meeting in L2, where an uneven split (full
// tiles and a short rest) lets them drift apart along K and fetch the panel
// from HBM again.  Tiles dealt round-robin or in groups over the XCDs start
// at multiples of bm (measured faster for the 256-row tiles, which run that
// way).
// Striped tiles (xcd_local == 2, n_tiles a multiple of 8, n_group 1) run
// in plain block order, so block L runs on XCD L % 8; within an expert,
// XCD x takes the n-tiles nt = x (mod 8), each with all its m-tiles in a row.
// Every XCD then streams an eighth of every expert's weights, and the m-tiles
// of one n-tile still share them in that XCD's L2.  With contiguous ranges per
// XCD, a skewed batch gives one XCD a single popular expert (many m-tiles,
// few weight bytes) and another many rare ones (few m-tiles each, many
// bytes); the tile counts match but the bytes to fetch do not.
template <class G>
__host__ __device__ __forceinline__ void tile_at(const G& g, int L, int bm, int bn, TileCoord& tc) {
  int lo = 0, hi = g.e_loc - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (g.tile_base[mid] * g.n_tiles <= L) lo = mid;
    else hi = mid - 1;
  }
  const int e = lo;
  const int mt_e = g.tile_base[e + 1] - g.tile_base[e];
  const int local = L - g.tile_base[e] * g.n_tiles;
  int mt, nt;
  if (g.xcd_local == 2) {
    const int j = local >> 3;
    const int q = j / mt_e;
    mt = j - q * mt_e;
    nt = 8 * q + (local & 7);
  } else {
    // Super-rows (m_super > 0): the expert's m-tiles are cut into runs of
    // m_super, each run taking all its n-tiles before the next (the last run
    // may be shorter); within a run the n-block order below applies.
    int m_base = 0, sm = mt_e, r0 = local;
    if (g.m_super > 0) {
      const int run = g.m_super * g.n_tiles;
      const int sr = local / run;
      m_base = sr * g.m_super;
      sm = min(g.m_super, mt_e - m_base);
      r0 = local - sr * run;
    }
    const int b = g.n_group;
    const int full = g.n_tiles / b;  // full n-blocks; a narrower one may follow
    int blk = r0 / (sm * b), bw = b;
    if (blk >= full) {
      blk = full;
      bw = g.n_tiles - full * b;
    }
    const int r = r0 - blk * sm * b;
    mt = m_base + r / bw;
    nt = blk * b + (r - (r / bw) * bw);
  }
  const int beg = g.offsets[e], rows = g.offsets[e + 1] - beg;
  const int per = (g.xcd_local == 1 || g.xcd_local == 2) ? (rows + mt_e - 1) / mt_e : bm;
  tc.e = e;
  tc.m0 = beg + mt * per;
  tc.m_end = min(tc.m0 + per, beg + rows);
  tc.n0 = nt * bn;
  tc.split = 0;
}

// Logical tile of this workgroup, or -1.  The dispatcher deals workgroups
// round-robin to the 8 XCDs; XCD x takes the logical tiles
// [x per_xcd, (x+1) per_xcd), so the tiles that share an expert's weights
// run side by side on one XCD's L2.  The grid, a multiple of 8 and at least
// the largest possible tile count, covers every tile.
//
// Grouped tiles (xcd_local == 3; the grid a multiple of 8 kXcdGroup): the
// logical tiles are cut into groups of kXcdGroup consecutive ids, one per
// XCD and round, dealt round-robin (group 8 r + x to XCD x in round r).  One
// round, 8 groups, is what the GPU runs at a time (one workgroup per CU), so
// every XCD works on the same expert as the others (whose bytes the
// memory-side cache then serves to all of them), and each XCD's own group is
// a compact block of tiles (with n_group 4: 8 m-tiles x 4 n-tiles), whose
// 8 row blocks and 4 weight panels its L2 serves to its 32 CUs.  Plain
// round-robin order gives each XCD 32 row blocks and one panel per round.
// The last round, when partial, is dealt round-robin tile by tile, so that
// every XCD takes a share of it.
constexpr int kXcdGroup = 32;  // workgroups one XCD runs at a time: one per CU

// Logical tile of the workgroup with block id b (see block_tile).
template <bool DENSE = false, class G>
__host__ __device__ __forceinline__ int tile_of_block(const G& g, int b) {
  int total;
  if constexpr (DENSE) total = g.dense_total;
  else total = g.tile_base[g.e_loc] * g.n_tiles;
  if (g.xcd_local == 3) {
    const int x = b & 7, slot = b >> 3;
    const int base = slot / kXcdGroup * (8 * kXcdGroup), j = slot % kXcdGroup;
    const int L = base + 8 * kXcdGroup <= total ? base + x * kXcdGroup + j : base + 8 * j + x;
    return L < total ? L : -1;
  }
  if (g.xcd_local != 1) return b < total ? b : -1;
  const int per_xcd = (total + 7) >> 3;
  const int slot = b >> 3;
  if (slot >= per_xcd) return -1;
  const int L = (b & 7) * per_xcd + slot;
  return L < total ? L : -1;
}

template <bool DENSE = false, class G>
__device__ __forceinline__ int block_tile(const G& g) {
  return tile_of_block<DENSE>(g, (int)blockIdx.x);
}

// D first (Section 3.1): the planner admits ready D work before P, and a
// long P execution is cut into segments so that D advances between them
// (Section 4.2).  On one GPU a segment is a run of K slices of a GEMM tile:
// while the other phase's layer window is open, a workgroup about to start a
// tile (and the LDS-ring tiles every few slices, see gemm_ring_body) sleeps
// in steps of 127 * 64 cycles until the window closes, at most `polls` times.
// The wait is bounded, so the kernel always finishes, and it is only a hint:
// no result depends on it.
// `budget` (polls left, wave-uniform) is shared by every wait of one tile,
// so a tile waits at most `polls` sleep steps in all, however long the
// window stays open.
__device__ __forceinline__ void yield_to_window(const YieldTo& y, int& budget) {
  if (!y.word) return;
  for (; budget > 0; --budget) {
    if (__hip_atomic_load(y.word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != y.gen) return;
    __builtin_amdgcn_s_sleep(127);
  }
}
__device__ __forceinline__ void yield_to_window(const YieldTo& y) {
  int budget = y.polls;
  yield_to_window(y, budget);
}

}  // namespace moepd
