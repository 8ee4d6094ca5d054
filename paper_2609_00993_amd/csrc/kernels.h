// Internal launch interface between the host runtime (ctx.hip) and the
// kernels.  Every launcher enqueues on the given stream and returns the
// hipError_t of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moepd {

// One phase's device buffers (owned by the context, see moepd.h).
struct PhaseBuffers {
  int32_t* topk_idx;      // [Tmax, k]
  float* topk_w;          // [Tmax, k]
  int32_t* counts;        // [E_loc]
  int32_t* offsets;       // [E_loc + 1]
  int32_t* row_of_slot;   // [Tmax, k]
  int32_t* token_of_row;  // [Rcap]
  void* x_perm;           // [Rcap, H]
  void* h;                // [Rcap, I]
  float* y;               // [Rcap, H] float32
  // workspace
  int32_t* chunk_counts;  // [E_loc * max_chunks], expert-major
  int32_t* tile_base;     // [E_loc + 1], prefix sum of m-tiles per expert
  // Signal word of this phase's layer window: a generation number while a
  // layer is between its route and its combine, 0 otherwise.  Written only
  // by this phase's kernels; read by the other phase's grouped GEMMs.  It is
  // the first word of a zeroed 16-byte slot (read as one 16-byte vector).
  int32_t* signal;
  // One word per tile of the 256-row GEMM2 run as a hand-over pair (see
  // launch_ffn_bf16): 1 = done by the first launch, cleared by the second.
  // Zero between layers.
  int32_t* tile_done;
  // router GEMM (moe_route_from_hidden)
  float* logits;    // [Tmax, E] float32, the logits top-k selects from
  float* partials;  // [router_cap_rows, E] float32, K-split partial products
};

// A layer window announced to the other phase: the kernels that open and
// close it store `gen` / 0 into `word` (null: no window).
struct WindowSignal {
  int32_t* word;
  int32_t gen;
};

// A window to yield to: a grouped-GEMM workgroup of the other phase waits
// while *word == gen, at most `polls` sleeps of about 3.4 us (null: never).
struct YieldTo {
  const int32_t* word;
  int32_t gen;
  int32_t polls;
};

// Largest number of (expert, chunk) histogram cells the count kernel scans.
constexpr int kMaxCells = 8192;
constexpr int kMaxTopK = 16;
constexpr int kMaxExperts = 1024;
constexpr int kMaxLocalExperts = 256;

// Batches of at most this many slots take one chunk: the place kernel then
// counts them itself and the count kernel is not launched (small D batches
// save a launch).
constexpr int kOneChunkSlots = 2048;

// Dispatch chunking: tokens per chunk for a batch of T tokens.
inline int dispatch_chunk_tokens(int T, int k, int e_loc) {
  if ((long long)T * k <= kOneChunkSlots) return T > 0 ? T : 1;
  int tc = (256 + k - 1) / k;
  int need = (int)(((long long)T * e_loc + kMaxCells - 1) / kMaxCells);
  if (need > tc) tc = need;
  return tc < 1 ? 1 : tc;
}

// Chunking of the dispatch histogram for T tokens: one chunk up to
// kOneChunkSlots slots, else about 256 slots per chunk, and never more than
// kMaxCells (expert, chunk) cells.
inline void dispatch_chunking(int T, int k, int e_loc, int* tc_out, int* nchunks_out) {
  int tc = dispatch_chunk_tokens(T, k, e_loc);
  int nc = T > 0 ? (T + tc - 1) / tc : 1;
  while ((long long)nc * e_loc > kMaxCells) {
    ++tc;
    nc = (T + tc - 1) / tc;
  }
  *tc_out = tc;
  *nchunks_out = nc < 1 ? 1 : nc;
}

// How the route kernel forms its logits after the router GEMM (out == null:
// read them as given).  logit[t][e] = sum over s < nsplit of
// in[(s T + t) E + e], in split order, + bias[e] (bias may be null); stored
// to out[t E + e] (out may equal in when nsplit == 1).
struct RouterSum {
  float* out;
  const float* bias;
  int nsplit;
};

hipError_t launch_route(const float* logits, int T, int E, int k, int32_t* topk_idx, float* topk_w,
                        WindowSignal open, RouterSum sum, hipStream_t s);

// Router GEMM (bf16, MFMA): partial logits of T tokens, out[s][t][e] =
// sum over split s's K run of x[t][h] w[e][h]; x [T, H] and w [E, H] bf16.
// router_splits picks the split count (and the slices per split, *ks) for a
// partial buffer of cap_rows rows (splits * T <= cap_rows).
int router_splits(int T, int E, int H, int cap_rows, int* ks);
hipError_t launch_router_bf16(const void* x, const void* w, int T, int E, int H, float* out, int splits, int ks,
                              YieldTo yield, hipStream_t s);
// Router GEMM (float32, vector ALUs): out[t][e] = sum_h x[t][h] w[e][h].
hipError_t launch_router_f32(const float* x, const float* w, int T, int E, int H, float* out, hipStream_t s);

// Histogram of each chunk's slots per local expert -> chunk_counts.
hipError_t launch_count(const int32_t* topk_idx, int T, int k, int e0, int e_loc, int chunk_tokens, int nchunks,
                        const PhaseBuffers& b, hipStream_t s);

// Scan of the histogram cells (block 0 publishes counts, offsets and the
// m-tile prefix for m-tiles of bm rows) and stable rows for every slot:
// row_of_slot and token_of_row.  Launched for every batch, T = 0 included.
// With one chunk (nchunks == 1) the kernel counts the slots itself and the
// count kernel is not launched.
hipError_t launch_place(const int32_t* topk_idx, int T, int k, int e0, int e_loc, int chunk_tokens, int nchunks,
                        int bm, const PhaseBuffers& b, hipStream_t s);

// x_perm[row] = x[t] for every resident slot (row-byte granularity 16 B).
hipError_t launch_permute(const void* x, int T, int k, int row_bytes, const int32_t* row_of_slot, void* x_perm,
                          hipStream_t s);

// Waves per token row in the permute and combine kernels: one for large
// batches (the rows alone fill the GPU); for small batches (up to 2048
// tokens) one per pass of 64 lanes x vec 16-byte vectors, so a token's passes
// run side by side instead of one after another.
inline int waves_per_row(int T, int nv, int vec) {
  if (T > 2048) return 1;
  const int pass = 64 * vec;
  return (nv + pass - 1) / pass;
}

// out[t] = sum_j w[t,j] y[row(t,j)] in float32 (y and out are float32).
hipError_t launch_combine(const void* y, const float* topk_w, const int32_t* row_of_slot, int T, int k, int H,
                          void* out, WindowSignal close, hipStream_t s);

// Grouped expert FFN.  `regime` picks the tile configuration (0 = large
// batches, 160-row tiles; 1 = small batches, 32-row weight-streaming tiles,
// one wave of 32 columns each; 2 = very large batches, 256-row tiles);
// ffn_bf16_bm gives its m-tile height, which the place kernel must use for
// tile_base.
int ffn_bf16_bm(int regime);
// stage (decode regime only): load operands as whole lines through a per-wave
// LDS stage (faster), or straight into registers with no LDS, so the tiles fit
// on CUs held by the other phase's 160-row prefill tiles.  share (256-row
// regime, GEMM2 only): the tiles that leave each CU room for the other
// phase's staged decode GEMM2 tiles (80 KB of LDS and 364 registers instead
// of 160 KB and 460; the same bits, 12 % slower alone) run only while the
// other phase has a layer in flight: a first launch of the full tiles does
// every tile that starts while `other_window` (the other phase's signal word)
// is 0 and marks it in b.tile_done, and a second launch of the share form
// does the rest.
hipError_t launch_ffn_bf16(int regime, int gemm, const PhaseBuffers& b, const void* w_gu, const void* w_dn,
                           int e_loc, int H, int I, int max_m_tiles, bool stage, bool share, YieldTo yield,
                           const int32_t* other_window, hipStream_t s);
// Words of b.tile_done a phase needs (256-row GEMM2 tiles at its capacity).
long long ffn_bf16_handover_words(long long rows_cap, int e_loc, int H);

// MX FP8 contexts: the phase's x_perm and h regions hold E4M3 codes
// followed by their E8M0 scale bytes (one per 32 values of a row).
struct MxBuffers {
  uint8_t* x_codes;   // [Rcap, H]
  uint8_t* x_scales;  // [Rcap, H / 32]
  uint8_t* h_codes;   // [Rcap, I]
  uint8_t* h_scales;  // [Rcap, I / 32]
};
struct MxWeights {
  const void* gu;         // [E_loc, 2I, H] E4M3 codes
  const void* gu_scales;  // [E_loc, 2I, H / 32] E8M0
  const void* dn;         // [E_loc, H, I] E4M3 codes
  const void* dn_scales;  // [E_loc, H, I / 32] E8M0
};
// x (bf16 rows) -> MX FP8 codes and scales of every resident row.
hipError_t launch_permute_mx(const void* x, int T, int k, int H, const int32_t* row_of_slot, uint8_t* codes,
                             uint8_t* scales, hipStream_t s);
// regime 0: large batches (256-row LDS-ring tiles); 1: small batches
// (32-row weight-streaming tiles).
int ffn_mx_bm(int regime);
hipError_t launch_ffn_mx(int regime, int gemm, const PhaseBuffers& b, const MxBuffers& mx, const MxWeights& w,
                         int e_loc, int H, int I, int max_m_tiles, YieldTo yield, hipStream_t s);

int ffn_f32_bm();
hipError_t launch_ffn_f32(int gemm, const PhaseBuffers& b, const void* w_gu, const void* w_dn, int e_loc, int H,
                          int I, int max_m_tiles, hipStream_t s);

}  // namespace moepd
