/*
 * moepd.h -- C ABI of libmoepd: one GPU's share of a DeepEP-style MoE expert
 * layer, run by a prefill (P) batch and a decode (D) batch concurrently on
 * shared weights, each phase owning its own mutable state.
 *
 * Paper: AInfer-PD, "Communication-Safe In-Place Prefill-Decode Multiplexing
 * for Distributed MoE Rollouts" (arXiv 2609.00993).
 *
 *  - Section 5.1 and its table "Ownership in the concurrent DeepEP runtime":
 *    P and D share runtime initialisation and model weights but each owns its
 *    buffers, counters, workspace, stream and events.  Here the context owns
 *    one such state set per phase; the weights are borrowed and shared.
 *  - Section 5.1 / Section 6 (first paragraph): phase identity selects state
 *    explicitly and is never inferred from a host thread or a stream, so every
 *    call below takes a phase id.  D keeps stable buffer addresses (captured
 *    graphs replay against them): all phase buffers are allocated once at
 *    context creation, at capacity.
 *  - Section 5.2: normal dispatch is split after expert notification, when
 *    the dispatch shape (per-expert counts) is known and before routed data
 *    moves.  moe_dispatch runs the notification part (histogram and prefix
 *    sum, the layout) and then the data movement (token permutation);
 *    moe_dispatch_layout and moe_dispatch_permute are the two halves, so a
 *    caller can stop at the boundary between them (a safe P boundary,
 *    Section 4.2) and let other work in before any routed data moves.
 *  - Section 5.2: at most one pending operation per phase buffer, with
 *    explicit transitions so that cancellation never reuses partially
 *    advanced state (the per-phase state machine and moe_phase_reset).
 *  - Section 5.3: an abandoned operation retires its buffer until a
 *    quiescent point (moe_phase_reset only succeeds once the phase's last
 *    enqueued work has completed).
 *  - Section 4.3 (idle ranks issue matched no-work calls): a batch of
 *    T = 0 tokens is legal and advances the phase like any other.
 *
 * The layer computed (the paper routes tokens to top-k experts, Section 7.1,
 * but leaves the layer's arithmetic to the engine): softmax over the expert
 * pool, top-k by logit with ties to the lower expert id (-0.0 == +0.0), the
 * k weights renormalised; slots routed outside the resident block
 * [e0, e0 + E_loc) are dropped from this GPU's share; the rows of an expert
 * are ordered by ascending token; expert e computes
 * y = (silu(x W1^T) * (x W3^T)) W2^T; out[t] = sum_j w[t,j] y[row(t,j)]
 * accumulated in float32 in slot order (zero when no slot is resident).
 * The config dtype is the type of the GEMM operands (x, weights, x_perm, h;
 * for FP8 contexts x is bf16 and the rest MX FP8, see MOE_DTYPE_FP8);
 * y and out are float32, the accumulation precision, in every context.
 *
 * Conventions
 *  - Every function returns MOE_OK (0) or a negative MOE_ERR_* code.
 *  - All argument and state validation happens on the host before anything
 *    is enqueued: a failing call enqueues nothing and changes no state.
 *  - State transitions happen at enqueue time, not at GPU completion.
 *  - Device pointers passed in are borrowed: the caller keeps them valid until
 *    the work enqueued on the given stream has completed.  Output buffers the
 *    caller passes are written by that work.
 *  - The library never synchronises a stream, never uses the null stream for
 *    work and never allocates after moe_ctx_create.  After each call it records
 *    the phase's event on the stream; if the next call on that phase comes on
 *    another stream, that stream first waits on the event.
 *  - Graph capture (Section 6.1: the D phase replays captured graphs against
 *    its stable buffers).  A phase's calls may be captured into a HIP graph
 *    on a stream the phase last ran on: while the stream captures, the
 *    library records no events and no timing, and a call arriving from
 *    another stream is refused with MOE_ERR_STATE.  The captured kernels
 *    carry the batch size and the argument pointers of the capture, and the
 *    enqueued work issues no memset.  Replays bypass the state machine: the
 *    caller orders them against the phase's other work and must not reset
 *    the phase while a replay is in flight.  After a moe_phase_reset, a D
 *    graph captured earlier no longer opens D-first windows that P honours.
 *  - One host thread may drive a phase at a time; P and D may be driven from
 *    different threads, because their host states are disjoint.
 *  - bf16 data is passed as uint16_t bit patterns (bfloat16), float32 as float.
 */
#ifndef MOEPD_H
#define MOEPD_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOEPD_ABI_VERSION 2

/* Phase ids. */
enum { MOE_PHASE_P = 0, MOE_PHASE_D = 1, MOE_NUM_PHASES = 2 };

/* Element type of x, the weights, x_perm and h (y and out are always float32).
 * MOE_DTYPE_FP8 (Section 7.1 runs FP8 checkpoints; the format is this
 * library's reading): x is bf16; the weights, x_perm and h are OCP MX FP8 --
 * E4M3 codes (one byte each) with one E8M0 scale byte per 32 consecutive
 * values of a row along K (value = E4M3(code) * 2^(scale - 127)).  x_perm and
 * h are quantized by the kernels: per 32 values of a row, the shared exponent
 * is floor(log2(max |v|)) - 8 (clamped to [-127, 127]; -127 for an all-zero
 * block) and each code is v / 2^exponent rounded to nearest even after
 * clamping to +-448.  H and I must be multiples of 128. */
enum { MOE_DTYPE_F32 = 0, MOE_DTYPE_BF16 = 1, MOE_DTYPE_FP8 = 2 };

/* Status codes. */
enum {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = -1,   /* bad configuration, null pointer, unsupported size */
  MOE_ERR_INVALID_PHASE = -2, /* phase id not MOE_PHASE_P or MOE_PHASE_D */
  MOE_ERR_CAPACITY = -3,      /* T above the phase's max_tokens */
  MOE_ERR_STATE = -4,         /* call out of order for the phase's state */
  MOE_ERR_BUSY = -5,          /* phase still has enqueued work in flight */
  MOE_ERR_OOM = -6,           /* device allocation failed at create */
  MOE_ERR_HIP = -7            /* a HIP runtime call failed */
};

/* Per-phase state machine: IDLE -route-> ROUTED -dispatch-> DISPATCHED
 * -expert_ffn-> COMPUTED -combine-> IDLE, where the dispatch step may be
 * taken in two: ROUTED -dispatch_layout-> LAID_OUT -dispatch_permute->
 * DISPATCHED. */
enum {
  MOE_STATE_IDLE = 0,
  MOE_STATE_ROUTED = 1,
  MOE_STATE_DISPATCHED = 2,
  MOE_STATE_COMPUTED = 3,
  MOE_STATE_LAID_OUT = 4
};

/* Kernels whose launches can be timed (moe_timing_*). */
enum {
  MOE_KERNEL_ROUTE = 0,   /* top-k gating */
  MOE_KERNEL_COUNT = 1,   /* per-chunk expert histogram (dispatch notification) */
  MOE_KERNEL_PLACE = 2,   /* prefix sum, counts/offsets and stable row assignment (dispatch layout) */
  MOE_KERNEL_PERMUTE = 3, /* token rows -> expert-contiguous rows (dispatch data movement) */
  MOE_KERNEL_GEMM1 = 4,   /* grouped gate/up GEMM with fused SwiGLU */
  MOE_KERNEL_GEMM2 = 5,   /* grouped down GEMM */
  MOE_KERNEL_COMBINE = 6, /* weighted gather-combine */
  MOE_KERNEL_ROUTER = 7,  /* router GEMM x Wr^T (moe_route_from_hidden) */
  MOE_NUM_KERNELS = 8
};

typedef struct moe_config {
  int32_t num_experts;       /* E: routed expert pool, 1..1024 */
  int32_t expert_begin;      /* e0: first resident expert, >= 0 */
  int32_t num_local_experts; /* E_loc: resident experts, 1..256, e0 + E_loc <= E */
  int32_t top_k;             /* k: 1..min(E, 16) */
  int32_t hidden;            /* H: multiple of 64 (of 128 for FP8), 64..16384 */
  int32_t inter;             /* I: multiple of 64 (of 128 for FP8), 64..16384 */
  int32_t dtype;             /* MOE_DTYPE_F32, MOE_DTYPE_BF16 or MOE_DTYPE_FP8 */
  int32_t max_tokens[MOE_NUM_PHASES]; /* capacity per phase, 0..1048576 */
  int32_t flags;             /* must be 0 */
  /* D-first admission, 0..1000 (0 = off).  Section 3.1: ready D work is
   * admitted before P, and a long P execution is cut into segments so that D
   * advances between them (Section 4.2).  On one GPU a P segment is a run of
   * K slices of one grouped-GEMM tile: while a D layer is in flight (from the
   * start of its moe_route kernel to the start of its moe_combine kernel), a P
   * grouped-GEMM workgroup about to start a tile, or at every fourth K slice
   * of a running tile, waits for the D layer, for at most about this many
   * microseconds per tile in all.  P's tiles of very large batches (256 rows,
   * at least 512 rows per expert expected) never wait, since each holds a
   * whole CU; once the context has run a D layer, a GEMM2 tile that starts
   * while a D layer is in flight takes a form that leaves its CU room for
   * D's tiles instead.  A scheduling hint only: results are unchanged. */
  int32_t d_priority_us;
} moe_config_t;

/* Borrowed, read-only expert weights for the E_loc resident experts, shared by
 * both phases (row-major, dtype of the config):
 *   w_gate_up [E_loc, 2I, H]: rows [0, I) = W1 (gate), rows [I, 2I) = W3 (up)
 *   w_down    [E_loc, H, I]:  W2
 * FP8 contexts pass E4M3 codes there and the E8M0 scale bytes in
 *   w_gate_up_scales [E_loc, 2I, H / 32], w_down_scales [E_loc, H, I / 32]
 * (scale b of a row covers its values [32 b, 32 b + 32)); other contexts
 * pass NULL.  They must stay valid for the context's lifetime. */
typedef struct moe_weights {
  const void* w_gate_up;
  const void* w_down;
  const void* w_gate_up_scales;
  const void* w_down_scales;
} moe_weights_t;

/* Device pointers and sizes of one phase's owned buffers (read-only for the
 * caller; contents are those left by the last completed call):
 *   topk_idx    [T, k] int32  global expert ids, slot j = j-th largest logit
 *   topk_w      [T, k] float  renormalised gate weights
 *   counts      [E_loc] int32 rows per resident expert
 *   offsets     [E_loc+1] int32 exclusive prefix sum of counts
 *   row_of_slot [T, k] int32  row of slot (t, j) in x_perm, -1 if dropped
 *   token_of_row[R]    int32  token of each row, R = offsets[E_loc]
 *   x_perm [R, H], h [R, I] in the config dtype; y [R, H] float32
 * Capacities: T <= max_tokens[phase], R <= rows_capacity. */
typedef struct moe_phase_view {
  int32_t state;
  int32_t tokens;        /* T of the batch in flight (last routed) */
  int32_t rows_capacity; /* max_tokens * min(k, E_loc) */
  int32_t reserved;
  int32_t* topk_idx;
  float* topk_w;
  int32_t* counts;
  int32_t* offsets;
  int32_t* row_of_slot;
  int32_t* token_of_row;
  void* x_perm;
  void* h;
  float* y;
  float* logits; /* [T, E] float32: the logits moe_route_from_hidden selected from */
  /* FP8 contexts: x_perm and h hold E4M3 codes ([R, H], [R, I] bytes) and
   * these their E8M0 scales ([R, H / 32], [R, I / 32]); NULL otherwise. */
  uint8_t* x_perm_scales;
  uint8_t* h_scales;
} moe_phase_view_t;

typedef struct moe_ctx moe_ctx_t;

/* Create a context on the current HIP device.  Validates cfg (see field
 * comments), allocates both phases' buffers at capacity (disjoint
 * allocations, fixed for the context's lifetime) and their events.  Creates no
 * stream.  Section 5.1 and its ownership table: the phases share the model
 * weights (here the borrowed w) and nothing a kernel writes; each phase owns
 * its buffers, counters, workspace and events, and D keeps stable addresses
 * for its captured graphs.  Errors: MOE_ERR_INVALID_ARG (null pointer, size out of range, k > E,
 * e0 + E_loc > E, flags != 0), MOE_ERR_OOM, MOE_ERR_HIP.  On error *out is
 * NULL and nothing is left allocated. */
int moe_ctx_create(const moe_config_t* cfg, const moe_weights_t* w, moe_ctx_t** out);

/* Top-k gating of T tokens (phase state IDLE -> ROUTED).
 * logits: borrowed device [T, E] float32, row-major, finite values.
 * Writes the phase's topk_idx and topk_w.  T = 0 is legal.
 * Errors: MOE_ERR_INVALID_ARG (null ctx; null logits with T > 0; T < 0),
 * MOE_ERR_INVALID_PHASE, MOE_ERR_CAPACITY, MOE_ERR_STATE, MOE_ERR_HIP. */
int moe_route(moe_ctx_t* ctx, int phase, const float* logits, int32_t T, hipStream_t stream);

/* Gating from hidden states (IDLE -> ROUTED): the router GEMM, then top-k.
 * logits[t][e] = sum_h x[t][h] w_router[e][h] (+ bias[e]), accumulated in
 * float32 (bf16 contexts multiply bf16 operands on the matrix cores; float32
 * contexts use float32 FMAs), stored in the phase's logits buffer
 * (moe_phase_view: logits); then the top-k gating of moe_route on exactly
 * those values.  The paper routes each token to its top-k experts (Section
 * 7.1); the gate's inputs are the token's hidden state.
 * x: borrowed device [T, H] in the config dtype, bf16 for FP8 contexts (the
 * rows moe_dispatch will move); w_router: borrowed device [E, H] in the same
 * type (bf16 for FP8 contexts), row e = expert
 * e's gate vector; bias: borrowed device [E] float32 or NULL.  bf16 contexts
 * may split the K (hidden) sum into runs added in a fixed order, so results
 * are deterministic.  Errors: MOE_ERR_INVALID_ARG (null x or w_router with
 * T > 0, T < 0, null stream), MOE_ERR_INVALID_PHASE, MOE_ERR_CAPACITY,
 * MOE_ERR_STATE, MOE_ERR_HIP. */
int moe_route_from_hidden(moe_ctx_t* ctx, int phase, const void* x, const void* w_router, const float* bias,
                          int32_t T, hipStream_t stream);

/* Dispatch (ROUTED -> DISPATCHED): the notification part computes counts,
 * offsets, row_of_slot and token_of_row (rows of an expert in ascending token
 * order, no padding); the data part copies x[t] into x_perm[row] for every
 * resident slot (FP8 contexts quantize each row to MX FP8 on the way, see
 * MOE_DTYPE_FP8).  x: borrowed device [T, H] in the config dtype, bf16 for
 * FP8 contexts (T from the
 * preceding moe_route).  Errors: MOE_ERR_INVALID_ARG (null x with T > 0),
 * MOE_ERR_INVALID_PHASE, MOE_ERR_STATE, MOE_ERR_HIP. */
int moe_dispatch(moe_ctx_t* ctx, int phase, const void* x, hipStream_t stream);

/* The notification half of moe_dispatch (ROUTED -> LAID_OUT, Section 5.2):
 * enqueues the histogram and the layout (counts, offsets, row_of_slot,
 * token_of_row) and moves no token data.  Once it returns the dispatch shape
 * is fixed on the stream; the phase may wait here, at a safe boundary, for as
 * long as the caller likes.  Errors: MOE_ERR_INVALID_ARG (null stream),
 * MOE_ERR_INVALID_PHASE, MOE_ERR_STATE, MOE_ERR_HIP. */
int moe_dispatch_layout(moe_ctx_t* ctx, int phase, hipStream_t stream);

/* The data half of moe_dispatch (LAID_OUT -> DISPATCHED): copies x[t] into
 * x_perm[row] for every resident slot, using the layout enqueued by
 * moe_dispatch_layout.  x as for moe_dispatch.  moe_dispatch_layout followed
 * by moe_dispatch_permute enqueues exactly the kernels of moe_dispatch.
 * Errors: MOE_ERR_INVALID_ARG (null x with T > 0, null stream),
 * MOE_ERR_INVALID_PHASE, MOE_ERR_STATE, MOE_ERR_HIP. */
int moe_dispatch_permute(moe_ctx_t* ctx, int phase, const void* x, hipStream_t stream);

/* Grouped expert FFN (DISPATCHED -> COMPUTED): h = silu(x_perm W1^T) *
 * (x_perm W3^T) and y = h W2^T for the rows of every resident expert: the
 * expert computation between DeepEP's dispatch and combine (Section 2.2; the
 * experts of the evaluated model, Section 7.1, in BF16 or FP8).  bf16
 * contexts multiply bf16 operands with float32 accumulation, round h to bf16
 * (nearest even; h is GEMM2's operand) and keep y in float32; float32
 * contexts compute everything in float32.  The tile schedule
 * is read from the device-side offsets (no host synchronisation).  bf16
 * small-batch tiles come in two forms with identical results: LDS-staged,
 * or, when the other phase's latest moe_expert_ffn ran large-batch tiles
 * (which leave too little LDS to share their CUs), register-direct; a
 * captured graph keeps the form chosen at capture.
 * Errors: MOE_ERR_INVALID_ARG, MOE_ERR_INVALID_PHASE, MOE_ERR_STATE, MOE_ERR_HIP. */
int moe_expert_ffn(moe_ctx_t* ctx, int phase, hipStream_t stream);

/* Weighted combine (COMPUTED -> IDLE): out[t] = sum over resident slots j, in
 * slot order, of topk_w[t,j] * y[row_of_slot[t,j]], accumulated in float32;
 * tokens with no resident slot get a zero row.  The receive side of DeepEP's
 * combine (Section 2.2) on this GPU's share of the experts: summing the
 * shares of all expert-parallel ranks gives the layer's output.
 * out: borrowed device [T, H] float32; every row is written.
 * Errors: MOE_ERR_INVALID_ARG (null out with T > 0), MOE_ERR_INVALID_PHASE,
 * MOE_ERR_STATE, MOE_ERR_HIP. */
int moe_combine(moe_ctx_t* ctx, int phase, void* out, hipStream_t stream);

/* Fill *view with the phase's buffer pointers and state: the phase-owned
 * objects of Section 5.1, read-only for the caller (parity checks, and the
 * stable addresses a captured D graph replays against, Section 6.1).
 * Errors: MOE_ERR_INVALID_ARG (null), MOE_ERR_INVALID_PHASE. */
int moe_phase_view(const moe_ctx_t* ctx, int phase, moe_phase_view_t* view);

/* Allocation-free dispatch layout, for callers that cannot allocate device
 * memory: code under graph capture, tight serving loops, harnesses that
 * forbid allocation.  It runs the kernels of moe_dispatch_layout on caller
 * buffers, with no context: from the routing indices it writes
 *   counts [E_loc], offsets [E_loc + 1], row_of_slot [T, k] (-1 = dropped)
 *   and token_of_row [R], R = offsets[E_loc] <= T * min(k, E_loc),
 * the same layout moe_dispatch_layout gives (rows of an expert in ascending
 * token order, no padding).
 * topk_idx: borrowed device [T, k] int32 global expert ids (as moe_route
 * writes them); expert_begin / num_local_experts: the resident block
 * [e0, e0 + E_loc).  All pointers are device pointers the caller owns, valid
 * until the work completes on `stream`; token_of_row must have room for
 * T * min(k, E_loc) entries.  T = 0 is legal (counts and offsets are zeroed).
 * It allocates nothing: the kernels' scratch (histogram cells and the m-tile
 * prefix, 33,796 bytes) is a fixed device array that each device holds until
 * the process ends, looked up on the first call on a device.  Every call on
 * a device shares that array, so calls that overlap on one device (other
 * streams or host threads) race and must be serialised by the caller.
 * Limits: T <= MOE_NOALLOC_MAX_TOKENS, 1 <= k <= 16, 1 <= E_loc <= 256.
 * Errors: MOE_ERR_INVALID_ARG (null pointer where T > 0 needs one, null
 * counts/offsets/stream, T < 0, k or E_loc out of range, e0 < 0),
 * MOE_ERR_CAPACITY (T above the limit), MOE_ERR_HIP.  A call refused for its
 * arguments enqueues nothing. */
#define MOE_NOALLOC_MAX_TOKENS (1 << 20)
int moe_dispatch_layout_noalloc(const int32_t* topk_idx, int32_t T, int32_t top_k, int32_t expert_begin,
                                int32_t num_local_experts, int32_t* counts, int32_t* offsets, int32_t* row_of_slot,
                                int32_t* token_of_row, hipStream_t stream);

/* Explicit transition back to IDLE (cancellation).  Succeeds only when every
 * operation enqueued for the phase has completed on the GPU; otherwise returns
 * MOE_ERR_BUSY and changes nothing.  Never touches the other phase.
 * Errors: MOE_ERR_INVALID_ARG, MOE_ERR_INVALID_PHASE, MOE_ERR_BUSY, MOE_ERR_HIP. */
int moe_phase_reset(moe_ctx_t* ctx, int phase);

/* Wait for both phases' enqueued work, then free every buffer and event the
 * context owns.  Never touches the borrowed weights.  NULL is a no-op. */
int moe_ctx_destroy(moe_ctx_t* ctx);

/* Static description of a status code (never NULL). */
const char* moe_status_string(int status);

/* ---- measurement aids ------------------------------------------------------
 * With timing enabled, every kernel launch of both phases is bracketed by a
 * pair of HIP events recorded on the stream the kernel is launched on.  Up to
 * max_launches launches are kept per (phase, kernel); later launches are not
 * timed.  Enabling allocates the events (call it before timed work);
 * max_launches = 0 disables timing and frees them.
 * Errors: MOE_ERR_INVALID_ARG, MOE_ERR_BUSY (work in flight), MOE_ERR_HIP. */
int moe_timing_enable(moe_ctx_t* ctx, int32_t max_launches);

/* Sum of the recorded launch durations (milliseconds) and their number for
 * one (phase, kernel), after waiting for the recorded events; then clears the
 * records.  Errors: MOE_ERR_INVALID_ARG, MOE_ERR_INVALID_PHASE, MOE_ERR_HIP. */
int moe_timing_read(moe_ctx_t* ctx, int phase, int kernel, double* total_ms, int32_t* launches);

/* Name of a MOE_KERNEL_* id ("?" when out of range). */
const char* moe_kernel_name(int kernel);

/* Engine clock probe.  One wave reads the shader-clock counter and the
 * 100 MHz reference counter, sleeps in short steps until spin_us
 * microseconds of the reference clock have passed (1..100000), and reads
 * both again.  out_dev: device memory for two uint64 values, written when
 * the kernel completes on `stream`: the shader-clock ticks and the
 * reference ticks of the spin, so the clock in MHz is out[0] * 100 / out[1].
 * Enqueued beside other work, it reads the clock under that load.  Uses no
 * context.  Errors: MOE_ERR_INVALID_ARG (null stream or pointer, spin_us
 * out of range), MOE_ERR_HIP. */
int moe_clock_probe(hipStream_t stream, int32_t spin_us, uint64_t* out_dev);

#ifdef __cplusplus
}
#endif

#endif /* MOEPD_H */
