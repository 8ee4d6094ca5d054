// Grouped expert FFN in bf16 on CDNA4 matrix cores (fp32 accumulation).
//
// GEMM1 (gated): for the rows [offsets[e], offsets[e+1]) of expert e,
//   h = silu(x_perm W1^T) * (x_perm W3^T), W1/W3 = rows [0,I)/[I,2I) of W_gu[e],
// with the SwiGLU applied in the epilogue so g and u never reach memory.
// GEMM2: y = h W2^T with W2 = W_dn[e].  h is rounded to bf16 (nearest even),
// the operand type of GEMM2; y stays float32, the accumulation precision.
// The paper's engine runs its own expert kernels (Section 7.1 states BF16 and
// FP8 checkpoints); this is a gfx950 design of the same contraction.
//
// Scheduling is fully device-side: the dispatch scan leaves tile_base, the
// prefix sum of m-tiles per expert, and each workgroup finds its tile from
// its id, so no host synchronisation is needed between dispatch and FFN.  The
// grid is an upper bound; surplus workgroups exit at once.  Tile ids run
// expert-major, then n-tile, then m-tile, and consecutive ids stay on one XCD
// (the dispatcher deals workgroups round-robin to the 8 XCDs): the m-tiles of
// one expert that share a weight tile run side by side on one XCD's L2.
//
// Three tile shapes, picked by the expected rows per expert:
//  * very large batches (at least 512 rows per expert): 256 x (128 gate +
//    128 up) or 256 x 256 tiles, a 2 x 2 grid of waves, 64-deep K slices in
//    two weight slots and three activation slots (160 KB), the activations
//    one slice ahead; GEMM2 also has a share form in 32-deep slices that
//    leaves a CU room for the other phase's decode tiles (gemm_ring_body and
//    the kernels below);
//  * large batches (prefill): 256 threads, 160 x (128 gate + 128 up) or
//    160 x 256 output tiles, 32x32x16 MFMAs, the four waves side by side
//    along N.  Operands stream HBM -> LDS with global_load_lds_dwordx4 into a
//    ring of three 64-deep K slices (156 KB); fragments are double-buffered
//    in registers and the LDS reads and DMA issues are interleaved with the
//    MFMAs (see gemm_ring_body).  160 rows, where 128 would be the plain
//    choice, because an expert's rows are shared evenly among its m-tiles:
//    with a few hundred rows per expert, ceil(rows / 160) saves the third,
//    mostly empty m-tile that ceil(rows / 128) adds whenever an expert holds
//    a little more than 256 rows, and every m-tile re-streams the weights;
//  * small batches (decode, a few rows per expert): the layer is a weight
//    stream, one 32-row m-tile and 32 columns per single-wave workgroup,
//    two 64-deep K blocks in flight.  Each block is loaded with whole-line
//    reads and transposed through the wave's own 12 KB LDS stage into MFMA
//    operand layout; beside the other phase's 160-row prefill tiles (which
//    leave 4 KB of LDS) the tile loads straight into operand registers
//    instead, with no LDS, so it can share their CUs.
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "tiles.h"
#include "pipeline.h"

namespace moepd {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct GemmArgs {
  const uint16_t* A;       // [R, K] expert-contiguous rows
  const uint16_t* B;       // expert e at B + e * b_stride, rows of length K
  void* C;                 // [R, N]: bf16 h (gated) or float32 y
  const int32_t* offsets;  // [E_loc + 1]
  const int32_t* tile_base;
  long long b_stride;
  int e_loc, N, K, n_tiles, up_row;
  int n_group;    // n-tiles per block of the within-expert tile order (see tile_at)
  int m_super;    // m-tiles per super-row of that order (0: one run over all of them)
  int xcd_local;  // 1: consecutive tiles on one XCD (block_tile); 0: dealt round-robin; 2: striped (tile_at)
  YieldTo yield;  // the other phase's layer window to hold back for, if any
  // Dense mode (the router GEMM): one group of dense_rows rows, no offsets;
  // K is cut into dense_splits runs of dense_ks slices and split s writes its
  // partial product to C + s * dense_rows * N.  dense_total = m-tiles x
  // n-tiles x splits.
  int dense_rows, dense_splits, dense_ks, dense_total;
  // Hand-over pair of the 256-row GEMM2 (see launch_ffn_bf16): 0 = off;
  // 1 = full tiles, a tile that starts while *window is nonzero is left to
  // the second launch; 2 = share tiles, a tile marked done is skipped.
  int handoff;
  const int32_t* window;
  int32_t* tile_done;
};

// First 64-deep K block of a decode tile (of nk blocks).  When a row of K
// bf16 values is a multiple of 4 KB (K % 2048 == 0), every weight row starts
// on the same memory channel, so tiles that stream the same K offset at the
// same time press on a few channels; rotating the start by the tile's
// (expert, n-tile) index spreads them.  Other pitches already spread and
// keep the plain order (the launch picks the variant), which measured faster
// for them.
__device__ __forceinline__ int k_rotation(const TileCoord& tc, int n_tiles, int bn, int nk) {
  return (int)((unsigned)((tc.e * n_tiles + tc.n0 / bn) * 2) % (unsigned)nk);
}

__device__ __forceinline__ bf16x8_t as_bf16x8(const u32x4& u) { return __builtin_bit_cast(bf16x8_t, u); }

// silu(g) * u for the bf16 h: the hardware reciprocal (about 1 ulp) is far
// inside the bf16 rounding of h and avoids an IEEE division per element.
__device__ __forceinline__ float silu_mul(float gt, float up) {
  return gt * __builtin_amdgcn_rcpf(1.f + __expf(-gt)) * up;
}

// Row i of the 32x32 accumulator element r held by `lane` (column = lane & 31).
__device__ __forceinline__ int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// ------------------------------------------------------------------ skinny (decode)

// Waves (32 output columns each) per decode workgroup.  One: every wave
// loads its own operands anyway, and with single-wave workgroups the tiles
// spread evenly over the CUs whatever their count (four-wave workgroups at
// 1.5 tiles per CU left half the CUs with two, which then set the pace).
constexpr int kDecodeWaves = 1;

template <bool GATED, bool ROT>
__device__ __forceinline__ void gemm_skinny_tile(const GemmArgs& g, const TileCoord& tc) {
  static_assert(kDecodeWaves == 1, "the LDS stage below is private to the workgroup's one wave");
  constexpr int BN = 32 * kDecodeWaves;
  constexpr int NB = GATED ? 2 : 1;
  constexpr int NP = 1 + NB;  // panels: the tile's activation rows, then its weight rows (gate, up)
  // A 64-deep K block of one panel is 32 rows x 128 B.  It is loaded as four
  // 1 KB instructions that each read eight whole 128-byte row pieces (lane
  // l: row 8i + l/8, 16-byte chunk l%8): reading 16 bytes from each of 32
  // rows per instruction, as the MFMA lane layout would, reaches only about a
  // quarter of the per-CU rate of whole-line reads.  The block then goes
  // through this wave's LDS stage, chunk c of row r at slot
  // 8r + (c ^ stage_swz(r)) (no bank conflicts on either side), and is read
  // back in the MFMA layout.
  __shared__ u32x4 stage[NP][32 * 8];
  const int lane = threadIdx.x & 63;
  const int lr = lane >> 3, lc = lane & 7;  // coalesced side: row within eight, chunk
  const int r = lane & 31, kg = lane >> 5;  // MFMA side
  const int col = tc.n0 + r;
  const uint16_t* Be = g.B + (size_t)tc.e * g.b_stride;
  const u32x4* base[NP];
  base[0] = reinterpret_cast<const u32x4*>(g.A);
  base[1] = reinterpret_cast<const u32x4*>(Be);
  if (GATED) base[NP - 1] = reinterpret_cast<const u32x4*>(Be + (size_t)g.up_row * g.K);
  const int kv = g.K / 8;  // 16-byte chunks per row
  // Chunk offset of this lane's row piece in block 0.  32 bits suffice: the
  // decode regime holds fewer than 32 rows per expert on average, so under
  // 32 x 1024 rows of at most 2048 chunks, and weight panels hold at most
  // 2 x 16384 rows.
  int off[NP][4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int rr = 8 * i + lr;
    off[0][i] = min(tc.m0 + rr, tc.m_end - 1) * kv + lc;
    const int cc = min(tc.n0 + rr, g.N - 1) * kv + lc;
#pragma unroll
    for (int j = 0; j < NB; ++j) off[1 + j][i] = cc;
  }
  int wslot[4];  // LDS slot of this lane's chunk for each of the four instructions
#pragma unroll
  for (int i = 0; i < 4; ++i) wslot[i] = (8 * i + lr) * 8 + (lc ^ stage_swz(8 * i + lr));
  // lane group kg holds k in [64*kb + 32*kg, +32) as four 16-byte chunks;
  // MFMA step s takes chunk s of both groups (the same k map for A and B).
  int rslot[4];
#pragma unroll
  for (int st = 0; st < 4; ++st) rslot[st] = r * 8 + ((4 * kg + st) ^ stage_swz(r));

  f32x16_t acc[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[j][q] = 0.f;

  const int KB = g.K / 64;
  const int krot = ROT ? k_rotation(tc, g.n_tiles, BN, KB) : 0;
  constexpr int PF = 2;  // 64-deep K blocks in flight per wave (a static register ring)
  u32x4 v[PF][NP][4];
  auto load = [&](int kb, u32x4 (&d)[NP][4]) {
    if (ROT) {
      kb += krot;
      if (kb >= KB) kb -= KB;
    }
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
      for (int i = 0; i < 4; ++i) d[p][i] = base[p][off[p][i] + kb * 8];
  };
#pragma unroll
  for (int q = 0; q < PF; ++q)
    if (q < KB) load(q, v[q]);
  for (int kb0 = 0; kb0 < KB; kb0 += PF) {
#pragma unroll
    for (int q = 0; q < PF; ++q) {
      const int kb = kb0 + q;
      if (kb < KB) {
        // LDS operations of one wave run in order, so these writes land after
        // the previous block's reads and before this block's.
#pragma unroll
        for (int p = 0; p < NP; ++p)
#pragma unroll
          for (int i = 0; i < 4; ++i) stage[p][wslot[i]] = v[q][p][i];
        if (kb + PF < KB) load(kb + PF, v[q]);
#pragma unroll
        for (int st = 0; st < 4; ++st) {
          const u32x4 a = stage[0][rslot[st]];
#pragma unroll
          for (int j = 0; j < NB; ++j)
            acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(stage[1 + j][rslot[st]]), acc[j],
                                                            0, 0, 0);
        }
      }
    }
  }

  if (col < g.N) {
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int row = tc.m0 + acc_row(q, lane);
      if (row < tc.m_end) {
        if (GATED)
          static_cast<uint16_t*>(g.C)[(size_t)row * g.N + col] = f32_to_bf16(silu_mul(acc[0][q], acc[NB - 1][q]));
        else
          static_cast<float*>(g.C)[(size_t)row * g.N + col] = acc[0][q];
      }
    }
  }
}

// The same tile with each operand loaded straight into MFMA lane layout (16
// bytes from each of 32 rows per instruction) and no LDS: slower alone, but
// it fits on a CU beside a 160-row prefill tile of the other phase, whose
// ring leaves 4 KB of LDS free.
template <bool GATED, bool ROT>
__device__ __forceinline__ void gemm_skinny_tile_direct(const GemmArgs& g, const TileCoord& tc) {
  constexpr int BN = 32 * kDecodeWaves;
  constexpr int NB = GATED ? 2 : 1;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 31, kg = lane >> 5;
  const int arow = min(tc.m0 + r, tc.m_end - 1);
  const int col = tc.n0 + wave * 32 + r;
  const int colc = min(col, g.N - 1);
  const uint16_t* Be = g.B + (size_t)tc.e * g.b_stride;
  // lane group kg holds k in [64*kb + 32*kg, +32) as four 16-byte chunks;
  // MFMA step s takes chunk s of both groups (the same k map for A and B).
  const u32x4* pa = reinterpret_cast<const u32x4*>(g.A + (size_t)arow * g.K) + kg * 4;
  const u32x4* pb[NB];
  pb[0] = reinterpret_cast<const u32x4*>(Be + (size_t)colc * g.K) + kg * 4;
  if (GATED) pb[NB - 1] = reinterpret_cast<const u32x4*>(Be + (size_t)(g.up_row + colc) * g.K) + kg * 4;

  f32x16_t acc[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[j][q] = 0.f;

  const int KB = g.K / 64;
  const int krot = ROT ? k_rotation(tc, g.n_tiles, BN, KB) : 0;
  constexpr int PF = 2;  // 64-deep K blocks in flight per wave (a static register ring)
  u32x4 ra[PF][4], rb[PF][NB][4];
  auto load = [&](int kb, u32x4 (&a)[4], u32x4 (&b)[NB][4]) {
    if (ROT) {
      kb += krot;
      if (kb >= KB) kb -= KB;
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      a[s] = pa[kb * 8 + s];
#pragma unroll
      for (int j = 0; j < NB; ++j) b[j][s] = pb[j][kb * 8 + s];
    }
  };
#pragma unroll
  for (int p = 0; p < PF; ++p)
    if (p < KB) load(p, ra[p], rb[p]);
  for (int kb0 = 0; kb0 < KB; kb0 += PF) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int kb = kb0 + p;
      if (kb < KB) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
          for (int j = 0; j < NB; ++j)
            acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(ra[p][s]), as_bf16x8(rb[p][j][s]), acc[j], 0, 0, 0);
        if (kb + PF < KB) load(kb + PF, ra[p], rb[p]);
      }
    }
  }

  if (col < g.N) {
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int row = tc.m0 + acc_row(q, lane);
      if (row < tc.m_end) {
        if (GATED)
          static_cast<uint16_t*>(g.C)[(size_t)row * g.N + col] = f32_to_bf16(silu_mul(acc[0][q], acc[NB - 1][q]));
        else
          static_cast<float*>(g.C)[(size_t)row * g.N + col] = acc[0][q];
      }
    }
  }
}

template <bool GATED, bool ROT, bool STAGE>
__device__ __forceinline__ void gemm_skinny(const GemmArgs& g) {
  constexpr int BM = 32, BN = 32 * kDecodeWaves;
  const int L = block_tile(g);
  if (L < 0) return;
  yield_to_window(g.yield);
  TileCoord tc;
  tile_at(g, L, BM, BN, tc);
  if constexpr (STAGE) gemm_skinny_tile<GATED, ROT>(g, tc);
  else gemm_skinny_tile_direct<GATED, ROT>(g, tc);
}

// One workgroup of 4 waves computes a BM x BN output tile of one expert.
// Per BK-deep K slice it stages A (BM rows) and B (BR weight rows: BN gate +
// BN up rows when GATED, BN rows otherwise) in LDS, swizzled as above.  The
// slices travel HBM -> LDS by global_load_lds_dwordx4 (lane l of an
// instruction lands 16 bytes at base + 16 l, so the swizzle is applied on the
// global side) into a ring of STAGES slots; no register or ds_write is spent
// on staging.
//
// The pipeline has three levels:
//  * DMA: once every wave has read slice kt out of its slot (the barrier at
//    the end of slice kt), slice kt + STAGES is issued into that slot, so
//    STAGES - 1 slices are in flight while one is multiplied.  The group goes
//    out in parts over the next slice's substeps (see PART_N).  Only this
//    wave's DMA instructions (and older stores) count in vmcnt, and loads
//    complete in order, so wait_vmcnt(n * per-slice count) retires exactly
//    the slices needed: every group is issued whole before the next begins;
//  * fragments: each 16-deep substep's A/B fragments are read from LDS into
//    one of two register sets while the MFMAs of the previous substep run on
//    the other (the read of a slice's first substep crosses the barrier);
//  * instructions: scheduling-group barriers spread the LDS reads and DMA
//    issues between the MFMAs, so the single wave per SIMD never waits on
//    its own reads.
//
// Wave (wm, wn) of the WM x WN wave grid owns rows [wm WTM, +WTM) and output
// columns [wn WTN, +WTN) (for GATED, the gate and the up column of the same
// index, so the SwiGLU is applied in registers).  The K loop is branch-free:
// rows past the expert's end are clamped to its last row and discarded at
// the store, which keeps the MFMA and LDS-read schedule intact.
// Slices between the in-tile checks of the D window (a power of two).
constexpr int kPauseEvery = 4;

// The D window word is read one check ahead by an LDS DMA issued after a
// slice's DMA: every lane lands the 16 bytes that start at the word (the
// phase's signal slot is 16 bytes) in its own 16-byte cell of one array the
// four waves share; all cells then hold a copy of the word.  The DMA is one
// more operation in the ring's queue: the counted waits at the slice ends
// retire it with the slices issued before the next one (waiting for one
// operation more than the slices need, never one less), so it has landed two
// slice ends later, and it is read back from LDS at the next check,
// kPauseEvery slices on.  A register load would either make the compiler
// wait for every outstanding DMA before its use (it cannot follow the count
// through the loop) or, untracked, leave a register the compiler may reuse
// while the load is still in flight.  Waves of one tile that read a cell while
// another wave's next DMA lands in it see the older or the newer copy; the
// word only steers a pause, and no result depends on it.  The LDS read is
// written out (with its own wait for LDS results) because the compiler,
// which tracks the 4-word DMA into this array, would otherwise wait for
// every outstanding DMA before it, draining the ring at each check; the
// counted waits have already retired the DMA it reads.
__device__ __forceinline__ int read_window_cell(const void* cell) {
  const uint32_t a = (uint32_t)(uintptr_t)MOEPD_LPTR(cell);
  int v;
  asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(a) : "memory");
  return v;
}
constexpr int kCachePolicyAgent = 0x10;  // sc1: coherent at agent scope

// STAGES slots hold weight slices; SA >= STAGES slots hold activation
// slices.  With SA = STAGES + 1 (two weight slots only) the activation
// slices run one slice further ahead than the weight slices: the slice end
// that issues B(j) is followed, over the next slice's substeps, by A(j + 1),
// so the counted wait at a slice end retires the next slice's weights while
// that slice's activations, issued a slice earlier, have had up to two
// slices' time to land.  WIN: the tile keeps the LDS cells of the D window
// word (tiles that never yield leave them out, which frees the LDS for the
// third activation slot).
template <int BM, int BR, int BK, int WM, int WN, bool GATED, int STAGES, bool DENSE = false, int SA = STAGES,
          bool WIN = true>
__device__ __forceinline__ void gemm_ring_body(const GemmArgs& g) {
  constexpr int NB = GATED ? 2 : 1;
  constexpr int BN = BR / NB;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 32, FN = WTN / 32, FB = FN * NB;
  constexpr int SUB = BK / 16;                     // MFMA K steps per slice
  constexpr int CPR = BK / 8;                      // 16-byte chunks per staged row
  constexpr int RPI = 64 / CPR;                    // rows per DMA instruction (1 KB)
  constexpr int A_INS = BM / RPI / 4, B_INS = BR / RPI / 4;  // per wave per slice
  constexpr int NPS = A_INS + B_INS;               // vector-memory ops per wave per slice
  constexpr int A_CH = BM * CPR, B_CH = BR * CPR;  // 16-byte chunks per slice
  constexpr int NRD = FM + FB, NMF = FM * FB;      // LDS reads and MFMAs per substep
  static_assert(WM * WN == 4, "four waves");
  static_assert(BK == 32 || BK == 64, "slice depth");
  static_assert(SUB % 2 == 0, "fragment double buffer alternates within a slice");
  static_assert(A_INS * RPI * 4 == BM && B_INS * RPI * 4 == BR, "slices split into whole DMA instructions");
  static_assert(FM * 32 == WTM && FN * 32 == WTN, "wave tile must be a multiple of 32x32");
  static_assert(STAGES >= 2 && NPS * (STAGES - 1) < 64, "pipeline depth");
  constexpr int LEAD = SA - STAGES;  // slices the activations run ahead of the weights
  static_assert(LEAD == 0 || (LEAD == 1 && STAGES == 2 && !WIN && !DENSE), "activation lead: two weight slots only");
  // The DMA group a slice end would issue goes out in parts, so the
  // vector-memory queue takes a part at a time beside the MFMAs instead of
  // the whole group at once.  Without the lead the group's NPS instructions
  // make SUB parts: the first at the slice end, the others one per substep
  // of the next slice (into the slot the barrier freed).  With it the
  // weights (one slice to land) go out whole at the slice end and the
  // activations' A_INS make SUB - 1 parts, one per substep of the next slice
  // but its last (their slot too was freed a barrier earlier).
  constexpr int PART_N = LEAD == 1 ? A_INS : NPS;       // instructions cut into parts
  constexpr int NPART = LEAD == 1 ? SUB - 1 : SUB;      // parts
  constexpr int END_PARTS = NPART - (SUB - 1);         // parts issued at the slice end (0 or 1)
  constexpr int PART0 = END_PARTS * PART_N / NPART;     // instructions among them
  static_assert(2 * A_INS + B_INS < 64, "prologue wait range");
  // One LDS object: the activation and weight rings of K slices, then (WIN)
  // the cells of the D window word (its first word in each cell, see
  // load_window).
  struct LdsRings {
    u32x4 a[SA][A_CH];
    u32x4 b[STAGES][B_CH];
  };
  struct LdsWin : LdsRings {
    u32x4 window[64];
  };
  __shared__ std::conditional_t<WIN, LdsWin, LdsRings> lds;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WN, wn = wave % WN;
  static_assert(!(DENSE && GATED), "the dense mode writes float32 partial products");
  int KT = g.K / BK;  // slices of this tile (a dense split takes its own run)
  // Per-lane DMA source rows: lane l fills LDS chunk l of its instruction,
  // row r = RPI i + l / CPR, physical chunk l % CPR, so it loads logical
  // chunk (l % CPR) ^ swz(r).
  const int lrow = lane / CPR, lphys = lane % CPR;

  // A rows are read through a buffer resource that covers exactly the
  // tile's rows of its expert: rows past the expert's end fall outside it,
  // so their loads return zeros and make no memory request (the output rows
  // they feed are never stored).  B rows past N are clamped to the last.
  __amdgpu_buffer_rsrc_t a_rsrc;
  uint32_t a_off[A_INS];  // byte offset of each A instruction's row chunk
  const uint16_t* b_src[B_INS];
  auto set_sources = [&](const TileCoord& tc) {
    const int m0 = __builtin_amdgcn_readfirstlane(tc.m0);
    const int rows = min(__builtin_amdgcn_readfirstlane(tc.m_end) - m0, BM);
    a_rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)(g.A + (size_t)m0 * g.K), (short)0, rows * g.K * 2,
                                               kBufferRsrcWord3);
    const uint16_t* Be = g.B + (size_t)__builtin_amdgcn_readfirstlane(tc.e) * g.b_stride;
    // first K element of the tile's run (a dense split starts further in)
    const int k0 = DENSE ? __builtin_amdgcn_readfirstlane(tc.split) * g.dense_ks * BK : 0;
#pragma unroll
    for (int i = 0; i < A_INS; ++i) {
      const int r = (wave * A_INS + i) * RPI + lrow;
      a_off[i] = (uint32_t)(r * g.K + k0 + (lphys ^ swz<BK>(r)) * 8) * 2u;
    }
#pragma unroll
    for (int i = 0; i < B_INS; ++i) {
      const int r = (wave * B_INS + i) * RPI + lrow;
      int brow;
      if (GATED) brow = r < BN ? min(tc.n0 + r, g.N - 1) : g.up_row + min(tc.n0 + r - BN, g.N - 1);
      else brow = min(tc.n0 + r, g.N - 1);
      b_src[i] = Be + (size_t)brow * g.K + k0 + (lphys ^ swz<BK>(r)) * 8;
    }
  };
  auto issue_a1 = [&](int i, int koff, int slot) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(a_rsrc, MOEPD_LPTR(&lds.a[slot][(wave * A_INS + i) * 64]), 16,
                                             a_off[i] + (uint32_t)koff * 2u, 0, 0, 0);
  };
  auto issue_b1 = [&](int i, int koff, int slot) {
    __builtin_amdgcn_global_load_lds(MOEPD_GPTR(b_src[i] + koff), MOEPD_LPTR(&lds.b[slot][(wave * B_INS + i) * 64]), 16,
                                     0, 0);
  };
  auto issue_a = [&](int kt, int slot) {
#pragma unroll
    for (int i = 0; i < A_INS; ++i) issue_a1(i, kt * BK, slot);
  };
  auto issue_b = [&](int kt, int slot) {
#pragma unroll
    for (int i = 0; i < B_INS; ++i) issue_b1(i, kt * BK, slot);
  };
  // Part p of slice kt's spread DMA into slot `slot`: instructions
  // [PART_N p / NPART, PART_N (p + 1) / NPART) of A's A_INS then B's B_INS
  // (with the lead, of A's alone).  p is a constant once the loops around a
  // call are unrolled, and so is every branch here.
  auto issue_part = [&](int kt, int slot, int p) {
#pragma unroll
    for (int i = PART_N * p / NPART; i < PART_N * (p + 1) / NPART; ++i) {
      if (LEAD == 1 || i < A_INS) issue_a1(i, kt * BK, slot);
      else issue_b1(i - A_INS, kt * BK, slot);
    }
  };
  // DMA group of slice j, whole (the prologue's): without a lead, A(j) then
  // B(j) into slot j % STAGES; with the activation lead, B(j) into weight
  // slot j % 2, then A(j + 1) (if the tile has it) into activation slot
  // (j + 1) % 3.
  auto issue = [&](int kt, int bslot, int aslot_next) {
    if constexpr (LEAD == 0) {
      issue_a(kt, bslot);
      issue_b(kt, bslot);
    } else {
      issue_b(kt, bslot);
      if (kt + 1 < KT) issue_a(kt + 1, aslot_next);
    }
  };
  auto load_window = [&] {
    if constexpr (WIN)
      __builtin_amdgcn_global_load_lds(MOEPD_GPTR(g.yield.word), MOEPD_LPTR(&lds.window[0]), 16, 0,
                                       kCachePolicyAgent);
  };
  auto prologue = [&](const TileCoord& tc) {
    set_sources(tc);
    if constexpr (LEAD == 1) issue_a(0, 0);
#pragma unroll
    for (int st = 0; st < STAGES; ++st)
      if (st < KT) issue(st, st, st + 1);
    if (WIN && g.yield.word) load_window();
  };

  bf16x8_t fa[2][FM], fb[2][FB];
  auto read_frags = [&](int aslot, int bslot, int sub, bf16x8_t (&a)[FM], bf16x8_t (&b)[FB]) {
    const u32x4* As = &lds.a[aslot][0];
    const u32x4* Bs = &lds.b[bslot][0];
    const int ch = 2 * sub + (lane >> 5);
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int r = wm * WTM + fm * 32 + (lane & 31);
      a[fm] = as_bf16x8(As[r * CPR + (ch ^ swz<BK>(r))]);
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        const int r = nb * BN + wn * WTN + fn * 32 + (lane & 31);
        b[nb * FN + fn] = as_bf16x8(Bs[r * CPR + (ch ^ swz<BK>(r))]);
      }
  };

  // The MFMAs take the weight fragment as their first operand, so each
  // accumulator holds a transposed 32x32 block: lane l owns output row
  // (l & 31) and, in registers 4q..4q+3, the four consecutive columns
  // 8q + 4 (l >> 5) + 0..3 (see the epilogue's vector stores).
  f32x16_t acc[FM][FB];
  auto mfmas = [&](const bf16x8_t (&a)[FM], const bf16x8_t (&b)[FB]) {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int j = 0; j < FB; ++j) acc[fm][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[j], a[fm], acc[fm][j], 0, 0, 0);
  };

  const int L = block_tile<DENSE>(g);
  if (L < 0) return;
  // Hand-over pair: one thread decides for the workgroup (whether the other
  // phase has a layer in flight now, or whether the first launch did this
  // tile) and passes the decision through the ring's first LDS word, which no
  // DMA has touched yet, so every wave leaves or stays together.
  constexpr bool HANDOFF = !GATED && !DENSE && BM == 256;
  if constexpr (HANDOFF) {
    if (g.handoff) {
      int* cell = reinterpret_cast<int*>(&lds);
      if (threadIdx.x == 0) {
        int skip;
        if (g.handoff == 1) {
          skip = __hip_atomic_load(g.window, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
        } else {
          skip = g.tile_done[L];
          if (skip) g.tile_done[L] = 0;
        }
        *cell = skip;
      }
      __syncthreads();
      const int skip = *cell;
      __syncthreads();  // every wave has read the word before the ring's DMA lands
      if (skip) return;
    }
  }
  int wait_budget = g.yield.polls;  // shared by the tile's start and in-tile waits
  yield_to_window(g.yield, wait_budget);
  TileCoord tc;
  if constexpr (DENSE) {
    dense_tile_at(g, L, BM, BN, tc);
    KT = min(g.dense_ks, KT - tc.split * g.dense_ks);
  } else {
    tile_at(g, L, BM, BN, tc);
  }
  prologue(tc);

#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FB; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Slice 0 has landed once at most min(STAGES - 1, KT - 1) newer slices
  // remain; with the activation lead, once at most A(1), B(1) and A(2) (those
  // the tile has) remain behind B(0).
  if constexpr (LEAD == 0) {
    wait_slices_lgkm0<NPS, STAGES - 1>(min(STAGES - 1, KT - 1));
  } else {
    if (KT > 2) wait_vmcnt_lgkm0<2 * A_INS + B_INS>();
    else if (KT == 2) wait_vmcnt_lgkm0<A_INS + B_INS>();
    else wait_vmcnt_lgkm0<0>();
  }
  bare_barrier();
  read_frags(0, 0, 0, fa[0], fb[0]);

  // One K slice.  MODE 0: slice kt + STAGES is issued into this slot after
  // the barrier; MODE 1: no slices left to issue; MODE 2: the tile's last
  // slice (no barrier, nothing to read ahead).  The three loops below keep
  // each body straight-line code, so the accumulators stay in place.
  // PEND: a group is still going out, one part per substep, into the slot
  // that the previous slice freed: parts 1 .. SUB - 1 of the group of slice
  // kt - 1 + STAGES (its part 0 went out at the previous slice end), or with
  // the lead all SUB - 1 parts of A(kt + 2) (B(kt + 1) went out whole there).
  auto slice = [&](auto mode, auto pend, int kt, int aslot, int bslot) {
    constexpr int MODE = decltype(mode)::value;
    constexpr bool PEND = decltype(pend)::value;
    int pkt, pslot;
    if constexpr (LEAD == 1) {
      pkt = kt + 2;
      pslot = aslot + 2 >= SA ? aslot + 2 - SA : aslot + 2;
    } else {
      pkt = kt - 1 + STAGES;
      pslot = bslot == 0 ? STAGES - 1 : bslot - 1;
    }
#pragma unroll
    for (int sub = 0; sub < SUB; ++sub) {
      const int cur = sub & 1, nxt = cur ^ 1;
      if (sub + 1 < SUB) {
        read_frags(aslot, bslot, sub + 1, fa[nxt], fb[nxt]);
        if constexpr (PEND) issue_part(pkt, pslot, END_PARTS + sub);
        mfmas(fa[cur], fb[cur]);
        interleave<0, NMF, PEND ? (PART_N + NPART - 1) / NPART : 0, NRD, 0>();
      } else if constexpr (MODE < 2) {
        // Every read of this slot is in registers once lgkmcnt is 0.  Slice
        // kt + 1 has landed once at most min(STAGES - 2, KT - 2 - kt) newer
        // slices remain; with the activation lead, once at most A(kt + 2)
        // (if the tile has it) remains behind B(kt + 1), A(kt + 1) having been
        // issued a group earlier.  After the barrier no wave reads this slot
        // again, so slice kt + STAGES (and A(kt + 3)) may overwrite it.
        if constexpr (LEAD == 1) {
          if (kt + 2 < KT) wait_vmcnt_lgkm0<A_INS>();
          else wait_vmcnt_lgkm0<0>();
        } else if constexpr (MODE == 0) {
          wait_vmcnt_lgkm0<NPS * (STAGES - 2)>();
        } else {
          wait_slices_lgkm0<NPS, STAGES - 2>(min(STAGES - 2, KT - 2 - kt));
        }
        bare_barrier();
        int nb = bslot + 1, na = aslot + 1;
        if (nb == STAGES) nb = 0;
        if (na == SA) na = 0;
        if constexpr (MODE == 0) {
          if constexpr (LEAD == 1) issue_b(kt + STAGES, bslot);
          else issue_part(kt + STAGES, bslot, 0);
          // D first inside a tile: every kPauseEvery slices, a P tile that
          // found the D window open at the previous check (or at the tile's
          // start) pauses until it closes (within the tile's wait budget), so
          // a D layer that starts while long P tiles run gets the memory
          // bandwidth.  The word read here was loaded into LDS one check
          // ahead, so its load never stalls the pipeline; its LDS read
          // completes before the next load into the same words is issued.
          if constexpr (WIN) {
            if (g.yield.word && (kt & (kPauseEvery - 1)) == kPauseEvery - 1) {
              const int seen = __builtin_amdgcn_readfirstlane(read_window_cell(&lds.window[lane]));
              if (seen == g.yield.gen) yield_to_window(g.yield, wait_budget);
              load_window();
            }
          }
        }
        read_frags(na, nb, 0, fa[nxt], fb[nxt]);
        mfmas(fa[cur], fb[cur]);
        interleave<0, NMF, MODE == 0 ? (LEAD == 1 ? B_INS : PART0) : 0, NRD, 1>();
      } else {
        mfmas(fa[cur], fb[cur]);
      }
    }
  };
  int kt = 0, aslot = 0, bslot = 0;
  auto advance = [&] {
    if (++bslot == STAGES) bslot = 0;
    if (++aslot == SA) aslot = 0;
  };
  using M0 = std::integral_constant<int, 0>;
  using M1 = std::integral_constant<int, 1>;
  using NoPend = std::false_type;
  using Pend = std::true_type;
  if (KT > STAGES) {
    // the prologue issued its groups whole: nothing pending in slice 0
    slice(M0{}, NoPend{}, kt, aslot, bslot);
    advance();
    for (++kt; kt < KT - STAGES; ++kt) {
      slice(M0{}, Pend{}, kt, aslot, bslot);
      advance();
    }
    // Without the lead, the group of slice KT - 1 (started at the last MODE-0
    // slice end) still goes out in the first MODE-1 slice; with it, the last
    // MODE-0 slice end issued B(KT - 1) alone, and nothing is pending.
    if constexpr (LEAD == 0) {
      slice(M1{}, Pend{}, kt, aslot, bslot);
      advance();
      ++kt;
    }
  }
  for (; kt < KT - 1; ++kt) {
    slice(M1{}, NoPend{}, kt, aslot, bslot);
    advance();
  }
  slice(std::integral_constant<int, 2>{}, NoPend{}, kt, aslot, bslot);

  // float32 y goes out through LDS (the ring is free once every wave has
  // read its last slice): each 32 x 32 block is written to the wave's own
  // LDS area in the accumulator layout, one 128-byte row per block row with
  // its 16-byte chunks XOR-swizzled by the row, and read back row-major, so
  // each store instruction writes eight whole 128-byte lines of y instead of
  // 32-byte pieces of 32 rows.  A block's 32 columns are all in range or all
  // out (N is a multiple of 64); rows past the expert's end are not stored.
  // Within a wave LDS operations complete in order, so a block's read-back
  // sees its writes and the next round's writes follow this round's reads.
  constexpr int NBLK = FM * FN;                                   // 32 x 32 blocks per wave
  constexpr int STAGE_BLK = sizeof(lds) / (4 * 4096);            // blocks one wave can stage
  constexpr int EPI_BLK = NBLK < STAGE_BLK ? NBLK : STAGE_BLK;   // per round (the last may hold fewer)
  constexpr bool STAGED_Y = !GATED && !DENSE && EPI_BLK > 0;
  if constexpr (STAGED_Y) {
    // every wave's reads of the ring are in registers (lgkmcnt 0; vmcnt is
    // already 0 after the last slice) before any wave overwrites it
    wait_vmcnt_lgkm0<63>();
    bare_barrier();
    u32x4* stage = reinterpret_cast<u32x4*>(&lds) + wave * (EPI_BLK * 256);
    const int wr = lane & 31, wh = lane >> 5;  // accumulator row, column half
    const int rr0 = lane >> 3, rc = lane & 7;  // read-back row (of 8), chunk
#pragma unroll
    for (int b0 = 0; b0 < NBLK; b0 += EPI_BLK) {
#pragma unroll
      for (int bi = 0; bi < EPI_BLK && b0 + bi < NBLK; ++bi) {
        const int fm = (b0 + bi) / FN, fn = (b0 + bi) % FN;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x4 v = {acc[fm][fn][4 * q], acc[fm][fn][4 * q + 1], acc[fm][fn][4 * q + 2],
                           acc[fm][fn][4 * q + 3]};
          stage[bi * 256 + wr * 8 + ((2 * q + wh) ^ (wr & 7))] = __builtin_bit_cast(u32x4, v);
        }
      }
#pragma unroll
      for (int bi = 0; bi < EPI_BLK && b0 + bi < NBLK; ++bi) {
        const int fm = (b0 + bi) / FN, fn = (b0 + bi) % FN;
        const int col0 = tc.n0 + wn * WTN + fn * 32;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const int rr = 8 * p + rr0;
          const u32x4 v = stage[bi * 256 + rr * 8 + (rc ^ (rr & 7))];
          const int row = tc.m0 + wm * WTM + fm * 32 + rr;
          if (row < tc.m_end && col0 < g.N)
            *reinterpret_cast<u32x4*>(static_cast<float*>(g.C) + (size_t)row * g.N + col0 + 4 * rc) = v;
        }
      }
    }
    if constexpr (HANDOFF) {
      if (g.handoff == 1 && threadIdx.x == 0) g.tile_done[L] = 1;
    }
    return;
  }

  // epilogue: SwiGLU -> bf16 h (four columns = one 8-byte store), or
  // float32 y (four columns = one 16-byte store).  A lane's row is fixed,
  // so it is checked once per 32-row block.  N is a multiple of 64, so a
  // four-column group is all in range or all out.
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int row = tc.m0 + wm * WTM + fm * 32 + (lane & 31);
    if (row >= tc.m_end) continue;
    if constexpr (DENSE) {
      // partial logits: float32, N (the expert count) need not be a
      // multiple of 4, so each column is checked
      float* Cs = static_cast<float*>(g.C) + ((size_t)tc.split * g.dense_rows + row) * g.N;
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int col = tc.n0 + wn * WTN + fn * 32 + 8 * q + 4 * (lane >> 5) + i;
            if (col < g.N) Cs[col] = acc[fm][fn][4 * q + i];
          }
      continue;
    }
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int col = tc.n0 + wn * WTN + fn * 32 + 8 * q + 4 * (lane >> 5);
        if (col >= g.N) continue;
        const size_t at = (size_t)row * g.N + col;
        if (GATED) {
          uint32_t lo = f32_to_bf16(silu_mul(acc[fm][fn][4 * q], acc[fm][FN + fn][4 * q]));
          lo |= (uint32_t)f32_to_bf16(silu_mul(acc[fm][fn][4 * q + 1], acc[fm][FN + fn][4 * q + 1])) << 16;
          uint32_t hi = f32_to_bf16(silu_mul(acc[fm][fn][4 * q + 2], acc[fm][FN + fn][4 * q + 2]));
          hi |= (uint32_t)f32_to_bf16(silu_mul(acc[fm][fn][4 * q + 3], acc[fm][FN + fn][4 * q + 3])) << 16;
          typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
          *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(g.C) + at) = u32x2{lo, hi};
        } else {
          f32x4 v = {acc[fm][fn][4 * q], acc[fm][fn][4 * q + 1], acc[fm][fn][4 * q + 2], acc[fm][fn][4 * q + 3]};
          *reinterpret_cast<f32x4*>(static_cast<float*>(g.C) + at) = v;
        }
      }
    }
  }
}

// Distinct entry points so that profiles name each GEMM of each regime.
__global__ __launch_bounds__(256) void gemm1_swiglu_prefill(GemmArgs g) { gemm_ring_body<160, 256, 64, 1, 4, true, 3>(g); }
__global__ __launch_bounds__(256) void gemm2_down_prefill(GemmArgs g) { gemm_ring_body<160, 256, 64, 1, 4, false, 3>(g); }
// The router GEMM: logits = x Wr^T over all T rows, 64 x 128 tiles, K split
// so that small batches still spread over the GPU.
__global__ __launch_bounds__(256) void router_gemm(GemmArgs g) { gemm_ring_body<64, 128, 64, 2, 2, false, 3, true>(g); }
// The wide tiles never yield (a P workgroup waiting on its CU would only keep
// D off it), so they leave out the window cells.  They take two weight slots
// and three activation slots, the activations one slice ahead and their DMA
// spread over the next slice's substeps, in 64-deep slices (160 KB; at the
// 16384-token skewed batch 4 % faster than 32-deep slices in four stages for
// GEMM1, 8 % for GEMM2).  GEMM2's share form takes 32-deep slices (80 KB,
// 364 registers), which leaves a CU room for D's staged GEMM2 tiles beside
// it: at that batch D's layer under P took 985 us against 1360-1400 us
// beside the 64-deep form (460 registers) and 1085 us beside a four-stage
// ring of 32-deep slices (128 KB).  Nothing of D's GEMM1 fits beside GEMM1's
// tile in either depth (456-460 registers).
__global__ __launch_bounds__(256) void gemm1_swiglu_wide(GemmArgs g) {
  gemm_ring_body<256, 256, 64, 2, 2, true, 2, false, 3, false>(g);
}
__global__ __launch_bounds__(256) void gemm2_down_wide(GemmArgs g) {
  gemm_ring_body<256, 256, 64, 2, 2, false, 2, false, 3, false>(g);
}
__global__ __launch_bounds__(256) void gemm2_down_wide_share(GemmArgs g) {
  gemm_ring_body<256, 256, 32, 2, 2, false, 2, false, 3, false>(g);
}
template <bool ROT, bool STAGE>
__global__ __launch_bounds__(64 * kDecodeWaves) void gemm1_swiglu_decode(GemmArgs g) {
  gemm_skinny<true, ROT, STAGE>(g);
}
template <bool ROT, bool STAGE>
__global__ __launch_bounds__(64 * kDecodeWaves) void gemm2_down_decode(GemmArgs g) {
  gemm_skinny<false, ROT, STAGE>(g);
}

// ------------------------------------------------------------------ launch

int ffn_bf16_bm(int regime) { return regime == 0 ? 160 : regime == 2 ? 256 : 32; }

static inline int round8(long long v) { return (int)((v + 7) / 8 * 8); }

long long ffn_bf16_handover_words(long long rows_cap, int e_loc, int H) {
  return (rows_cap / 256 + 1 + e_loc) * (long long)((H + 255) / 256);
}

hipError_t launch_ffn_bf16(int regime, int gemm, const PhaseBuffers& b, const void* w_gu, const void* w_dn,
                           int e_loc, int H, int I, int max_m_tiles, bool stage, bool share, YieldTo yield,
                           const int32_t* other_window, hipStream_t s) {
  GemmArgs g{};
  g.yield = yield;
  g.offsets = b.offsets;
  g.tile_base = b.tile_base;
  g.e_loc = e_loc;
  if (gemm == 1) {
    g.A = (const uint16_t*)b.x_perm;
    g.B = (const uint16_t*)w_gu;
    g.C = b.h;
    g.b_stride = 2LL * I * H;
    g.N = I;
    g.K = H;
    g.up_row = I;
  } else {
    g.A = (const uint16_t*)b.h;
    g.B = (const uint16_t*)w_dn;
    g.C = b.y;
    g.b_stride = (long long)H * I;
    g.N = H;
    g.K = I;
    g.up_row = 0;
  }
  if (regime == 0 || regime == 2) {
    g.n_tiles = gemm == 1 ? (g.N + 127) / 128 : (g.N + 255) / 256;
    // 160-row tiles (a few m-tiles per expert): the m-tiles of one n-tile
    // run together on one XCD and share its weights in that XCD's L2.
    // 256-row tiles (large experts, many m-tiles): tiles are dealt to the
    // XCDs in groups (block_tile), so the whole GPU works through one expert
    // at a time and the expert's bytes stay in the memory-side cache, while
    // each XCD takes blocks of 8 m-tiles x 4 n-tiles whose row blocks and
    // weight panels its L2 shares.
    g.n_group = regime == 2 ? 4 : 1;
    g.xcd_local = regime == 2 ? 3 : 1;
    // GEMM1's 256-row tiles go through an expert in super-rows of as many
    // m-tiles as one round of the grid (8 XCDs x kXcdGroup tiles) covers
    // with all n-tiles: 16 m-tiles x 16 n-tiles at I = 2048.  Each round then
    // reads each of its activation blocks once, where rounds of all the
    // expert's m-tiles x 4 n-tiles re-read every block (3.7 MB each at
    // H = 7168) once per block of n-tiles, more than the memory-side cache
    // keeps for a popular expert (16384 rows: 235 MB): 3 % faster at the
    // 16384-token skewed batch.  GEMM2's row blocks (1 MB at I = 2048) stay
    // cached and its tiles keep the plain order, which measured faster.
    g.m_super = regime == 2 && gemm == 1 ? (8 * kXcdGroup + g.n_tiles - 1) / g.n_tiles : 0;
    const long long tiles = (long long)max_m_tiles * g.n_tiles;
    const dim3 grid(regime == 2 ? (int)((tiles + 8 * kXcdGroup - 1) / (8 * kXcdGroup) * (8 * kXcdGroup))
                                : round8(tiles));
    if (regime == 0) {
      if (gemm == 1) gemm1_swiglu_prefill<<<grid, 256, 0, s>>>(g);
      else gemm2_down_prefill<<<grid, 256, 0, s>>>(g);
    } else {
      if (gemm == 1) {
        gemm1_swiglu_wide<<<grid, 256, 0, s>>>(g);
      } else if (share && other_window) {
        // the full tiles while the other phase is idle, then the share form
        // for the tiles they left (the second launch follows the first on
        // the stream, so it sees every mark)
        g.window = other_window;
        g.tile_done = b.tile_done;
        g.handoff = 1;
        gemm2_down_wide<<<grid, 256, 0, s>>>(g);
        g.handoff = 2;
        gemm2_down_wide_share<<<grid, 256, 0, s>>>(g);
      } else if (share) {
        gemm2_down_wide_share<<<grid, 256, 0, s>>>(g);
      } else {
        gemm2_down_wide<<<grid, 256, 0, s>>>(g);
      }
    }
  } else {
    constexpr int bn = 32 * kDecodeWaves, threads = 64 * kDecodeWaves;
    g.n_tiles = (g.N + bn - 1) / bn;
    g.n_group = 1;
    g.m_super = 0;
    g.xcd_local = g.n_tiles % 8 == 0 ? 2 : 1;
    const dim3 grid(round8((long long)max_m_tiles * g.n_tiles));
    const bool rot = g.K % 2048 == 0;
    auto go = [&](auto k) { k<<<grid, threads, 0, s>>>(g); };
    if (gemm == 1) {
      if (stage) rot ? go(gemm1_swiglu_decode<true, true>) : go(gemm1_swiglu_decode<false, true>);
      else rot ? go(gemm1_swiglu_decode<true, false>) : go(gemm1_swiglu_decode<false, false>);
    } else {
      if (stage) rot ? go(gemm2_down_decode<true, true>) : go(gemm2_down_decode<false, true>);
      else rot ? go(gemm2_down_decode<true, false>) : go(gemm2_down_decode<false, false>);
    }
  }
  return hipGetLastError();
}

// K splits of the router GEMM: enough tiles x splits to cover the GPU twice,
// at most 16 splits (the top-k kernel adds them up) and at least 4 slices
// per split (a split has a three-slice pipeline to fill).
int router_splits(int T, int E, int H, int cap_rows, int* ks_out) {
  const int tiles = ((T + 63) / 64) * ((E + 127) / 128);
  const int kt = H / 64;
  int s = (512 + tiles - 1) / tiles;
  s = s < 16 ? s : 16;
  s = s < kt / 4 ? s : kt / 4;
  const int by_cap = T > 0 ? cap_rows / T : 1;
  s = s < by_cap ? s : by_cap;
  if (s < 1) s = 1;
  const int ks = (kt + s - 1) / s;
  *ks_out = ks;
  return (kt + ks - 1) / ks;
}

hipError_t launch_router_bf16(const void* x, const void* w, int T, int E, int H, float* out, int splits, int ks,
                              YieldTo yield, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  GemmArgs g{};
  g.A = (const uint16_t*)x;
  g.B = (const uint16_t*)w;
  g.C = out;
  g.offsets = nullptr;
  g.tile_base = nullptr;
  g.b_stride = 0;
  g.e_loc = 1;
  g.N = E;
  g.K = H;
  g.up_row = 0;
  g.n_tiles = (E + 127) / 128;
  g.n_group = g.n_tiles;
  g.m_super = 0;
  g.xcd_local = 0;
  g.yield = yield;
  g.dense_rows = T;
  g.dense_splits = splits;
  g.dense_ks = ks;
  g.dense_total = ((T + 63) / 64) * g.n_tiles * splits;
  router_gemm<<<dim3(round8(g.dense_total)), 256, 0, s>>>(g);
  return hipGetLastError();
}

}  // namespace moepd
