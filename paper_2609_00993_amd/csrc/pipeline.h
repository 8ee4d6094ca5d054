// Building blocks of the LDS-ring GEMMs (bf16 and MX FP8): counted waits on
// this wave's vector-memory operations, the fence-free workgroup barrier,
// the LDS row swizzle, the instruction-interleaving hints, and the raw
// buffer-resource word used for bounds-checked DMA.
#pragma once

#include <hip/hip_runtime.h>

namespace moepd {

// Word 3 of a raw (unstructured) buffer resource on gfx9: 32-bit data
// format, no swizzle; out-of-range loads return zero without a memory access.
constexpr int kBufferRsrcWord3 = 0x00020000;

#define MOEPD_GPTR(p) ((const void __attribute__((address_space(1)))*)(p))
#define MOEPD_LPTR(p) ((void __attribute__((address_space(3)))*)(p))

// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding:
// vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8], vmcnt[5:4] in bits [15:14]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

// Wait until at most `newer` slices of NPS DMA instructions each are in
// flight (newer <= MAXN, wave-uniform).
template <int NPS, int MAXN>
__device__ __forceinline__ void wait_slices(int newer) {
  if constexpr (MAXN > 0) {
    if (newer >= MAXN) {
      wait_vmcnt<NPS * MAXN>();
      return;
    }
    wait_slices<NPS, MAXN - 1>(newer);
  } else {
    wait_vmcnt<0>();
  }
}

// The swizzle depends on the row length.
// A staged row is BK bf16 = 2 BK bytes = CPR 16-byte chunks, and 256 / (2 BK)
// rows share one 256-byte sweep of the 64 LDS banks.  Chunk c of row r is
// stored at c ^ swz(r), swz(r) = (r / rows_per_sweep) % CPR, so the 16 lanes
// that a ds_read_b128 serves together (16 consecutive rows, one chunk each)
// cover all 64 banks once.
template <int BK>
__device__ __forceinline__ int swz(int row) {
  constexpr int CPR = BK / 8, RPS = 256 / (2 * BK);
  return (row / RPS) & (CPR - 1);
}

// Swizzle of the small-batch tiles' per-wave LDS stage: a 64-deep K block of
// 32 rows, chunk c (16 bytes) of row r at slot 8 r + (c ^ stage_swz(r)).  A
// 16-lane group of the whole-line writes covers two rows, which share the
// swizzle, so it writes 256 consecutive bytes; a 16-lane group of the MFMA
// reads takes one chunk of 16 consecutive rows, whose slots then fall on
// (r % 2, stage_swz(r)) = 16 different 16-byte bank groups.  (Swizzling by
// r % 8 put rows r and r + 8 on the same banks: two-way conflicts.)
__device__ __forceinline__ int stage_swz(int row) { return (row >> 1) & 7; }

// Workgroup barrier without a memory fence; the signal fences keep the
// compiler from moving LDS accesses across it.  Visibility of the DMA'd
// stages is established by wait_vmcnt before the barrier.
__device__ __forceinline__ void bare_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// s_waitcnt vmcnt(n) lgkmcnt(0): this wave's LDS reads are done and at most
// n of its vector-memory operations are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x70);
}

template <int NPS, int MAXN>
__device__ __forceinline__ void wait_slices_lgkm0(int newer) {
  if constexpr (MAXN > 0) {
    if (newer >= MAXN) {
      wait_vmcnt_lgkm0<NPS * MAXN>();
      return;
    }
    wait_slices_lgkm0<NPS, MAXN - 1>(newer);
  } else {
    wait_vmcnt_lgkm0<0>();
  }
}

// Scheduling-group masks of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedMfma = 0x008, kSchedVmem = 0x010, kSchedDsRead = 0x100;

// Ask the scheduler for N MFMAs with NR LDS reads spread over the first half
// of them (so the reads have the second half to land before the next
// substep needs them) and NV vector-memory instructions over the second
// half (sync group SYNC).
template <int I, int N, int NV, int NR, int SYNC>
__device__ __forceinline__ void interleave() {
  if constexpr (I < N) {
    constexpr int H = (N + 1) / 2;
    __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, SYNC);
    if constexpr (I < H) {
      constexpr int r = NR * (I + 1) / H - NR * I / H;
      if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, r, SYNC);
    } else {
      constexpr int v = NV * (I - H + 1) / (N - H) - NV * (I - H) / (N - H);
      if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(kSchedVmem, v, SYNC);
    }
    interleave<I + 1, N, NV, NR, SYNC>();
  }
}

}  // namespace moepd
