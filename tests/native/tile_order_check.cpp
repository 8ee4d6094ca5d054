// Host check of the grouped GEMMs' tile scheduler (csrc/tiles.h): for the
// launch shapes the library uses, every workgroup id of the grid maps to at
// most one logical tile, every logical tile to exactly one workgroup, every
// (expert, m-tile, n-tile) appears once, and each expert's m-tiles cover its
// rows [offsets[e], offsets[e+1]) without overlap, none longer than the tile
// height and none empty, for every n-tile.  Shapes: the 256-row tiles dealt
// to the XCDs in groups (GEMM1 in super-rows of one grid round, GEMM2 in the
// plain order), the 160-row tiles with the rows shared evenly, and the
// 32-row decode tiles (striped over the XCDs or in contiguous ranges), over
// random and skewed row counts and the edges (empty experts, one row, exact
// multiples of the tile height).
//
// Built with hipcc for the host only; prints "ok" and exits 0 when every
// check holds.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "tiles.h"

using namespace moepd;

struct G {
  const int32_t* offsets;
  const int32_t* tile_base;
  int e_loc, n_tiles, n_group, m_super, xcd_local;
  int dense_rows, dense_splits, dense_ks, dense_total;
};

static int failures = 0;
#define CHECK(cond, ...)                   \
  do {                                     \
    if (!(cond)) {                         \
      if (failures < 20) {                 \
        std::printf("FAIL %s: ", #cond);   \
        std::printf(__VA_ARGS__);          \
        std::printf("\n");                 \
      }                                    \
      ++failures;                          \
    }                                      \
  } while (0)

// One launch: rows per expert, tile height bm, n-tiles, the order fields,
// and the grid the launcher would use.
static void check_launch(const std::vector<int>& rows, int bm, int n_tiles, int n_group, int m_super, int xcd_local,
                         const char* what) {
  const int e_loc = (int)rows.size();
  std::vector<int32_t> off(e_loc + 1, 0), tb(e_loc + 1, 0);
  long long R = 0;
  for (int e = 0; e < e_loc; ++e) {
    off[e + 1] = off[e] + rows[e];
    tb[e + 1] = tb[e] + (rows[e] + bm - 1) / bm;
    R += rows[e];
  }
  G g{off.data(), tb.data(), e_loc, n_tiles, n_group, m_super, xcd_local, 0, 0, 0, 0};
  const long long total = (long long)tb[e_loc] * n_tiles;
  // the launchers' grids: an upper bound on the tiles from the row count
  const long long max_m_tiles = (R + bm - 1) / bm + e_loc;
  const long long tiles = max_m_tiles * n_tiles;
  long long grid;
  if (xcd_local == 3) grid = (tiles + 8 * kXcdGroup - 1) / (8 * kXcdGroup) * (8 * kXcdGroup);
  else grid = (tiles + 7) / 8 * 8;
  CHECK(grid >= total, "%s: grid %lld < %lld tiles", what, grid, total);
  std::vector<int> seenL(total, 0);
  // per (expert, n-tile): row coverage counts
  std::vector<std::vector<int>> cover(n_tiles, std::vector<int>(R > 0 ? R : 1, 0));
  std::vector<int> seen_coord;  // (tile index within expert) per expert x n
  std::vector<std::vector<int>> mt_seen(e_loc);
  for (int e = 0; e < e_loc; ++e) mt_seen[e].assign((size_t)(tb[e + 1] - tb[e]) * n_tiles, 0);
  for (long long b = 0; b < grid; ++b) {
    const int L = tile_of_block(g, (int)b);
    if (L < 0) continue;
    CHECK(L < total, "%s: block %lld -> tile %d of %lld", what, b, L, total);
    if (L >= total) continue;
    ++seenL[L];
    TileCoord tc;
    tile_at(g, L, bm, 32, tc);
    CHECK(tc.e >= 0 && tc.e < e_loc, "%s: tile %d expert %d", what, L, tc.e);
    if (tc.e < 0 || tc.e >= e_loc) continue;
    const int beg = off[tc.e], end = off[tc.e + 1];
    CHECK(tc.m0 >= beg && tc.m_end <= end && tc.m0 < tc.m_end, "%s: tile %d rows [%d,%d) outside [%d,%d)", what, L,
          tc.m0, tc.m_end, beg, end);
    CHECK(tc.m_end - tc.m0 <= bm, "%s: tile %d holds %d rows > %d", what, L, tc.m_end - tc.m0, bm);
    const int nt = tc.n0 / 32;
    CHECK(tc.n0 % 32 == 0 && nt >= 0 && nt < n_tiles, "%s: tile %d n0 %d", what, L, tc.n0);
    if (nt < 0 || nt >= n_tiles) continue;
    for (int r = tc.m0; r < tc.m_end && r < end; ++r) ++cover[nt][r];
  }
  for (long long L = 0; L < total; ++L) CHECK(seenL[L] == 1, "%s: tile %lld taken %d times", what, L, seenL[L]);
  for (int nt = 0; nt < n_tiles; ++nt)
    for (long long r = 0; r < R; ++r)
      CHECK(cover[nt][r] == 1, "%s: n-tile %d row %lld covered %d times", what, nt, r, cover[nt][r]);
}

int main() {
  std::mt19937 rng(7);
  std::vector<std::vector<int>> cases;
  // the skewed layer's shape: 32 experts, capped-Zipf rows (a few of ~16k)
  {
    std::vector<int> r(32);
    for (int e = 0; e < 32; ++e) r[e] = (int)(16384.0 * 0.125 / (e < 2 ? 1.0 : 0.64 * (e + 1) * 0.8)) + (e * 37) % 91;
    cases.push_back(r);
  }
  // uniform-ish, ragged
  for (int t = 0; t < 6; ++t) {
    std::vector<int> r(1 + rng() % 40);
    for (auto& v : r) v = (int)(rng() % 1200);
    cases.push_back(r);
  }
  // edges: empty experts, one row, exact multiples of 32/160/256
  cases.push_back({0, 1, 0, 256, 512, 160, 320, 32, 0});
  cases.push_back({1});
  cases.push_back({4097, 0, 0, 2303, 2398});
  cases.push_back({0, 0, 0});
  int launches = 0;
  for (const auto& rows : cases) {
    for (int n_tiles : {1, 2, 3, 16, 28, 32, 64}) {
      // 256-row tiles, grouped over the XCDs: GEMM1 with super-rows of one
      // round, GEMM2 in the plain order
      const int ms = (8 * kXcdGroup + n_tiles - 1) / n_tiles;
      check_launch(rows, 256, n_tiles, 4, ms, 3, "wide super-rows");
      check_launch(rows, 256, n_tiles, 4, 0, 3, "wide plain");
      check_launch(rows, 256, n_tiles, 8, 5, 3, "wide odd super-rows");
      // 160-row tiles, consecutive tiles on one XCD, rows shared evenly
      check_launch(rows, 160, n_tiles, 1, 0, 1, "prefill");
      // 32-row decode tiles: striped when the n-tiles are a multiple of 8
      check_launch(rows, 32, n_tiles, 1, 0, n_tiles % 8 == 0 ? 2 : 1, "decode");
      launches += 5;
    }
  }
  if (failures) {
    std::printf("%d failures\n", failures);
    return 1;
  }
  std::printf("%d launches checked\nok\n", launches);
  return 0;
}
