/*
 * moepd_turnstile.h -- host-side segment turnstile of libmoepd: lets D
 * iterations in between segments of a long P execution at safe P boundaries,
 * and a P-epoch runner that drives a context's P phase through it.
 *
 * Paper: AInfer-PD, "Communication-Safe In-Place Prefill-Decode Multiplexing
 * for Distributed MoE Rollouts" (arXiv 2609.00993).
 *
 *  - Section 4.2 (rank-aligned segment boundaries): a P epoch e carries
 *    boundary ids i = 0, 1, ... published in increasing order by exactly one
 *    producer.  The controller keeps the largest reached boundary r (-1 at
 *    the start of an epoch), the permitted endpoint p, a positive span K and
 *    the task state.  P stops at i = p; after each D iteration an active P
 *    task gets p <- p + K.  p starts at 0 when a ready D has not been
 *    enqueued yet (D goes first, before P touches the GPU) and at K when D is
 *    already enqueued.  The controller refuses stale or duplicate epochs,
 *    publications with no registered producer, boundaries that do not
 *    increase, and boundaries beyond the current permit.
 *  - Section 4.3 (the turnstile step).  P: wait before any GPU work while
 *    p = 0; publish each boundary; after publishing i, wait while i >= p;
 *    report TaskDone after the final segment.  D: if p > 0, wait until
 *    r >= p or TaskDone; enqueue the D iteration; then release the next
 *    segment (p <- p + K) without waiting for any GPU completion.
 *  - Section 4.3 (the two rendezvous): with one GPU and one process there is
 *    one participant, so the pre-D and post-D rendezvous are the controller's
 *    own lock; they carry no value and wait for no GPU event, as there.
 *  - Section 5.2: the backend's boundary is the point after dispatch
 *    notification and before routed data movement; the P-epoch runner below
 *    publishes boundary l after moe_dispatch_layout of layer l and moves the
 *    layer's data (moe_dispatch_permute) only once permitted.
 *  - Section 6.2: the segment policy chooses the span; moe_turnstile_set_span
 *    changes it between rounds without changing the ordering rules.
 *
 * Conventions
 *  - Every function returns MOE_OK (0) or a negative status code
 *    (moe_status_string describes each).  A refused call changes no state and
 *    is counted in moe_turnstile_state_t.rejected.
 *  - Host-only: nothing here touches the GPU except the P-epoch runner, which
 *    enqueues the P phase's kernels through the moepd.h calls.
 *  - Thread safety: every moe_turnstile_* call may be made from any thread;
 *    the intended use is one P thread (the producer) and one D thread.  The
 *    two waits block on a condition variable with a timeout.
 */
#ifndef MOEPD_TURNSTILE_H
#define MOEPD_TURNSTILE_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#include "moepd.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Further status codes (see moepd.h for the others). */
enum {
  MOE_ERR_REJECTED = -8, /* turnstile refused the call (stale or duplicate epoch, no producer,
                            boundary not increasing or beyond the permit, release without entry) */
  MOE_ERR_TIMEOUT = -9   /* a turnstile wait or the P-epoch runner ran out of time */
};

/* Task state of the current epoch. */
enum { MOE_TS_IDLE = 0, MOE_TS_ACTIVE = 1, MOE_TS_DONE = 2 };

/* Kinds of logged transitions (moe_turnstile_event_t.kind). */
enum {
  MOE_TS_EV_BEGIN = 0,   /* value = initial permit p */
  MOE_TS_EV_PUBLISH = 1, /* value = boundary i */
  MOE_TS_EV_RESUME = 2,  /* P passed its wait; value = boundary it waited at (-1: before the GPU) */
  MOE_TS_EV_ENTER = 3,   /* D passed its wait (pre-D phase); value = p at that moment */
  MOE_TS_EV_RELEASE = 4, /* D released the next segment (post-D phase); value = new p */
  MOE_TS_EV_DONE = 5     /* TaskDone; value = r at that moment */
};

typedef struct moe_turnstile_state {
  int64_t epoch;      /* current epoch, -1 before the first */
  int64_t reached;    /* r: largest published boundary of the epoch (-1: none) */
  int64_t permit;     /* p: permitted endpoint */
  int32_t span;       /* K applied at the next release */
  int32_t task;       /* MOE_TS_IDLE / ACTIVE / DONE */
  int64_t rounds;     /* releases while the epoch's task was active */
  int64_t rejected;   /* refused calls since creation */
  double p_wait_us;   /* time the current epoch's P spent in moe_turnstile_wait_permit */
  double d_wait_us;   /* time D spent in moe_turnstile_wait_boundary during the current epoch */
  int64_t d_entries;  /* D entries during the current epoch */
  int64_t log_dropped; /* events not logged because the log was full */
} moe_turnstile_state_t;

typedef struct moe_turnstile_event {
  int32_t kind;  /* MOE_TS_EV_* */
  int32_t reserved;
  int64_t epoch;
  int64_t value; /* see the kinds */
  int64_t t_ns;  /* steady-clock time of the transition, nanoseconds */
} moe_turnstile_event_t;

typedef struct moe_turnstile moe_turnstile_t;

/* Create a controller with span K = span (>= 1) and room for log_capacity
 * logged events (0 .. 1 << 20; 0 disables the log).  No epoch is active.
 * Errors: MOE_ERR_INVALID_ARG (null out, span < 1, capacity out of range),
 * MOE_ERR_OOM.  On error *out is NULL. */
int moe_turnstile_create(int32_t span, int32_t log_capacity, moe_turnstile_t** out);

/* Free the controller.  No thread may be inside a call on it.  NULL is a no-op. */
int moe_turnstile_destroy(moe_turnstile_t* ts);

/* Set K for the releases that follow (segment policy, Section 6.2).
 * Errors: MOE_ERR_INVALID_ARG (null, span < 1). */
int moe_turnstile_set_span(moe_turnstile_t* ts, int32_t span);

/* Register the producer of P epoch `epoch` (Section 4.2): r = -1, p = K if
 * d_enqueued (the ready D is already enqueued) else 0, task ACTIVE; the
 * per-epoch wait counters restart.  Refused (MOE_ERR_REJECTED) when epoch is
 * not above every epoch begun before (stale or duplicate) or the current
 * epoch is still ACTIVE.  Errors: MOE_ERR_INVALID_ARG (null), MOE_ERR_REJECTED. */
int moe_turnstile_begin(moe_turnstile_t* ts, int64_t epoch, int32_t d_enqueued);

/* P publishes boundary `boundary` of `epoch` (r = boundary) and wakes D.
 * Refused when no producer is registered for epoch (not the current epoch or
 * its task not ACTIVE), when boundary <= r (not increasing; duplicates
 * included), when boundary > p, or while p = 0 (P may not have started).
 * Errors: MOE_ERR_INVALID_ARG (null, boundary < 0), MOE_ERR_REJECTED. */
int moe_turnstile_publish(moe_turnstile_t* ts, int64_t epoch, int64_t boundary);

/* P's wait.  boundary = -1: the wait before any GPU work, passes once p > 0.
 * boundary >= 0: must be the last published boundary (r); passes once
 * boundary < p.  Blocks up to timeout_us microseconds (0: test only).
 * Errors: MOE_ERR_INVALID_ARG (null, boundary < -1, timeout_us < 0),
 * MOE_ERR_REJECTED (epoch not current and ACTIVE, boundary >= 0 and != r),
 * MOE_ERR_TIMEOUT (still not permitted; the state is unchanged). */
int moe_turnstile_wait_permit(moe_turnstile_t* ts, int64_t epoch, int64_t boundary, int64_t timeout_us);

/* TaskDone for epoch (after the final segment): task DONE, wakes D.
 * Errors: MOE_ERR_INVALID_ARG (null), MOE_ERR_REJECTED (epoch not current and ACTIVE). */
int moe_turnstile_done(moe_turnstile_t* ts, int64_t epoch);

/* D's wait (pre-D phase).  Passes at once when no task is ACTIVE or p = 0,
 * else once r >= p or the task is done.  On success D is inside: it enqueues
 * its iteration and then calls moe_turnstile_release.  Blocks up to
 * timeout_us microseconds (0: test only).
 * Errors: MOE_ERR_INVALID_ARG (null, timeout_us < 0), MOE_ERR_REJECTED (D is
 * already inside), MOE_ERR_TIMEOUT. */
int moe_turnstile_wait_boundary(moe_turnstile_t* ts, int64_t timeout_us);

/* D's release (post-D phase): when the task is ACTIVE and was already ACTIVE
 * when D entered, p <- p + K and P is woken; otherwise nothing moves (a D
 * that entered before the epoch began is the enqueued D that begin's
 * d_enqueued accounts for).  Never waits.
 * Errors: MOE_ERR_INVALID_ARG (null), MOE_ERR_REJECTED (D is not inside). */
int moe_turnstile_release(moe_turnstile_t* ts);

/* Snapshot of the controller.  Errors: MOE_ERR_INVALID_ARG (null). */
int moe_turnstile_query(moe_turnstile_t* ts, moe_turnstile_state_t* out);

/* Move up to `capacity` logged events, oldest first, into out (caller-owned
 * array) and drop them from the log; *count receives the number moved.
 * Errors: MOE_ERR_INVALID_ARG (null ts or count, capacity < 0, null out with
 * capacity > 0). */
int moe_turnstile_log(moe_turnstile_t* ts, moe_turnstile_event_t* out, int32_t capacity, int32_t* count);

/* ---- P-epoch runner --------------------------------------------------------
 * Runs one P epoch of `layers` MoE layers on the P phase of ctx from a host
 * thread of its own, through the turnstile ts: it begins epoch `epoch`
 * (moe_turnstile_begin with d_enqueued), waits before its first launch, and
 * for each layer l enqueues moe_route and moe_dispatch_layout, publishes
 * boundary l and waits for the permit, then enqueues moe_dispatch_permute,
 * moe_expert_ffn and moe_combine; it reports TaskDone after the last layer.
 * Layer l reads logits[l] (device [T, E] float32) and x[l] (device [T, H],
 * config dtype) and writes out[l] (device [T, H] float32): host arrays of
 * `layers` device pointers, copied at start (the same pointer may repeat).
 * The device buffers are borrowed until the enqueued work completes.
 * Every wait is bounded by timeout_us.  On any failure the runner stops
 * enqueueing, reports TaskDone (so D never waits on it) and returns the
 * failing status from moe_p_epoch_join; the P phase is then left in the
 * state the failing call found (moe_phase_reset after the stream drains).
 * The P phase must be IDLE and not be driven by another thread meanwhile. */
typedef struct moe_p_epoch_stats {
  int32_t status;        /* status of the epoch (MOE_OK or the first error) */
  int32_t layers_done;   /* layers fully enqueued */
  double enqueue_us;     /* host time spent enqueueing (waits excluded) */
  double wait_us;        /* host time spent waiting for permits */
  int64_t t_begin_ns;    /* steady clock: epoch begun */
  int64_t t_end_ns;      /* steady clock: last call returned */
} moe_p_epoch_stats_t;

typedef struct moe_p_runner moe_p_runner_t;

/* Start the runner.  Errors (nothing started): MOE_ERR_INVALID_ARG (null
 * pointer, layers < 1, T < 0, timeout_us < 1, null logits/x/out entries with
 * T > 0), MOE_ERR_STATE (P phase not IDLE), MOE_ERR_REJECTED (the turnstile
 * refuses the epoch), MOE_ERR_OOM. */
int moe_p_epoch_start(moe_ctx_t* ctx, moe_turnstile_t* ts, int64_t epoch, int32_t d_enqueued, int32_t layers,
                      int32_t T, const float* const* logits, const void* const* x, float* const* out,
                      hipStream_t stream, int64_t timeout_us, moe_p_runner_t** runner);

/* Wait for the runner's thread, fill *stats (may be NULL) and free the
 * runner.  Returns the epoch's status.  Errors: MOE_ERR_INVALID_ARG (null runner). */
int moe_p_epoch_join(moe_p_runner_t* runner, moe_p_epoch_stats_t* stats);

#ifdef __cplusplus
}
#endif

#endif /* MOEPD_TURNSTILE_H */
