// Segment turnstile (Sections 4.2-4.3) and the P-epoch runner that drives a
// context's P phase through it, publishing one boundary per layer after the
// dispatch notification (Section 5.2).  Host code only.
//
// The controller is one mutex-protected record (epoch, r, p, K, task) with a
// condition variable for the two waits.  With a single participant the
// paper's pre-D and post-D rendezvous reduce to taking the lock: D enters
// only when P has stopped at its permitted endpoint (or finished), and P
// resumes only after D's release has moved the endpoint.
#include <algorithm>
#include <chrono>
#include <condition_variable>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "moepd_turnstile.h"

namespace {

using Clock = std::chrono::steady_clock;

int64_t now_ns() {
  return std::chrono::duration_cast<std::chrono::nanoseconds>(Clock::now().time_since_epoch()).count();
}

constexpr int32_t kMaxLog = 1 << 20;

}  // namespace

struct moe_turnstile {
  std::mutex mu;
  std::condition_variable cv;
  int64_t highest = -1;  // highest epoch ever begun
  int64_t epoch = -1;
  int64_t r = -1, p = 0;
  int32_t span = 1;
  int32_t task = MOE_TS_IDLE;
  bool d_inside = false;
  bool d_in_epoch = false;  // D entered while epoch d_epoch was active
  int64_t d_epoch = -1;
  int64_t rounds = 0, rejected = 0, d_entries = 0, dropped = 0;
  double p_wait_us = 0.0, d_wait_us = 0.0;
  std::vector<moe_turnstile_event_t> log;  // ring of `cap` events
  int32_t cap = 0, head = 0, count = 0;

  // Caller holds mu.
  void note(int32_t kind, int64_t value) {
    if (cap == 0) return;
    if (count == cap) {
      ++dropped;
      return;
    }
    log[(head + count) % cap] = moe_turnstile_event_t{kind, 0, epoch, value, now_ns()};
    ++count;
  }
  int reject() {
    ++rejected;
    return MOE_ERR_REJECTED;
  }
  bool active(int64_t e) const { return task == MOE_TS_ACTIVE && e == epoch; }
  // D may enter: no active task, p = 0 (target 0 needs no publication), or P
  // has reached the endpoint.
  bool d_may_enter() const { return task != MOE_TS_ACTIVE || p == 0 || r >= p; }
};

namespace {

// Wait on ts->cv until pred() holds or timeout_us passes; returns whether it
// holds.  Adds the time spent to *acc.
template <typename Pred>
bool wait_for(moe_turnstile* ts, std::unique_lock<std::mutex>& lk, int64_t timeout_us, double* acc, Pred pred) {
  if (pred()) return true;
  if (timeout_us == 0) return false;
  const auto t0 = Clock::now();
  // Bounded at one hour so that the deadline cannot overflow the clock.
  const int64_t us = std::min<int64_t>(timeout_us, 3600ll * 1000 * 1000);
  const bool ok = ts->cv.wait_for(lk, std::chrono::microseconds(us), pred);
  *acc += std::chrono::duration<double, std::micro>(Clock::now() - t0).count();
  return ok;
}

}  // namespace

extern "C" {

int moe_turnstile_create(int32_t span, int32_t log_capacity, moe_turnstile_t** out) {
  if (!out) return MOE_ERR_INVALID_ARG;
  *out = nullptr;
  if (span < 1 || log_capacity < 0 || log_capacity > kMaxLog) return MOE_ERR_INVALID_ARG;
  moe_turnstile* ts = new (std::nothrow) moe_turnstile();
  if (!ts) return MOE_ERR_OOM;
  try {
    ts->log.resize((size_t)log_capacity);
  } catch (const std::bad_alloc&) {
    delete ts;
    return MOE_ERR_OOM;
  }
  ts->cap = log_capacity;
  ts->span = span;
  *out = ts;
  return MOE_OK;
}

int moe_turnstile_destroy(moe_turnstile_t* ts) {
  delete ts;
  return MOE_OK;
}

int moe_turnstile_set_span(moe_turnstile_t* ts, int32_t span) {
  if (!ts || span < 1) return MOE_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(ts->mu);
  ts->span = span;
  return MOE_OK;
}

int moe_turnstile_begin(moe_turnstile_t* ts, int64_t epoch, int32_t d_enqueued) {
  if (!ts) return MOE_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(ts->mu);
  if (epoch <= ts->highest || ts->task == MOE_TS_ACTIVE) return ts->reject();
  ts->highest = ts->epoch = epoch;
  ts->r = -1;
  ts->p = d_enqueued ? ts->span : 0;
  ts->task = MOE_TS_ACTIVE;
  ts->rounds = ts->d_entries = 0;
  ts->p_wait_us = ts->d_wait_us = 0.0;
  ts->note(MOE_TS_EV_BEGIN, ts->p);
  ts->cv.notify_all();
  return MOE_OK;
}

int moe_turnstile_publish(moe_turnstile_t* ts, int64_t epoch, int64_t boundary) {
  if (!ts || boundary < 0) return MOE_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(ts->mu);
  if (!ts->active(epoch) || boundary <= ts->r || boundary > ts->p || ts->p == 0) return ts->reject();
  ts->r = boundary;
  ts->note(MOE_TS_EV_PUBLISH, boundary);
  ts->cv.notify_all();
  return MOE_OK;
}

int moe_turnstile_wait_permit(moe_turnstile_t* ts, int64_t epoch, int64_t boundary, int64_t timeout_us) {
  if (!ts || boundary < -1 || timeout_us < 0) return MOE_ERR_INVALID_ARG;
  std::unique_lock<std::mutex> lk(ts->mu);
  if (!ts->active(epoch) || (boundary >= 0 && boundary != ts->r)) return ts->reject();
  // The epoch cannot change under the wait: only its own producer could end it.
  const bool ok = wait_for(ts, lk, timeout_us, &ts->p_wait_us,
                           [&] { return boundary < 0 ? ts->p > 0 : boundary < ts->p; });
  if (!ok) return MOE_ERR_TIMEOUT;
  ts->note(MOE_TS_EV_RESUME, boundary);
  return MOE_OK;
}

int moe_turnstile_done(moe_turnstile_t* ts, int64_t epoch) {
  if (!ts) return MOE_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(ts->mu);
  if (!ts->active(epoch)) return ts->reject();
  ts->task = MOE_TS_DONE;
  ts->note(MOE_TS_EV_DONE, ts->r);
  ts->cv.notify_all();
  return MOE_OK;
}

int moe_turnstile_wait_boundary(moe_turnstile_t* ts, int64_t timeout_us) {
  if (!ts || timeout_us < 0) return MOE_ERR_INVALID_ARG;
  std::unique_lock<std::mutex> lk(ts->mu);
  if (ts->d_inside) return ts->reject();
  const bool ok = wait_for(ts, lk, timeout_us, &ts->d_wait_us, [&] { return ts->d_may_enter(); });
  if (!ok) return MOE_ERR_TIMEOUT;
  ts->d_inside = true;
  ts->d_in_epoch = ts->task == MOE_TS_ACTIVE;
  ts->d_epoch = ts->epoch;
  ++ts->d_entries;
  ts->note(MOE_TS_EV_ENTER, ts->p);
  return MOE_OK;
}

int moe_turnstile_release(moe_turnstile_t* ts) {
  if (!ts) return MOE_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(ts->mu);
  if (!ts->d_inside) return ts->reject();
  ts->d_inside = false;
  // Only a D that entered during this epoch moves its permit: the D that
  // was already inside when the epoch began is the one p = K accounted for.
  if (ts->task == MOE_TS_ACTIVE && ts->d_in_epoch && ts->d_epoch == ts->epoch) {
    ts->p += ts->span;
    ++ts->rounds;
  }
  ts->note(MOE_TS_EV_RELEASE, ts->p);
  ts->cv.notify_all();
  return MOE_OK;
}

int moe_turnstile_query(moe_turnstile_t* ts, moe_turnstile_state_t* out) {
  if (!ts || !out) return MOE_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(ts->mu);
  out->epoch = ts->epoch;
  out->reached = ts->r;
  out->permit = ts->p;
  out->span = ts->span;
  out->task = ts->task;
  out->rounds = ts->rounds;
  out->rejected = ts->rejected;
  out->p_wait_us = ts->p_wait_us;
  out->d_wait_us = ts->d_wait_us;
  out->d_entries = ts->d_entries;
  out->log_dropped = ts->dropped;
  return MOE_OK;
}

int moe_turnstile_log(moe_turnstile_t* ts, moe_turnstile_event_t* out, int32_t capacity, int32_t* count) {
  if (!ts || !count || capacity < 0 || (capacity > 0 && !out)) return MOE_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(ts->mu);
  const int32_t n = std::min(capacity, ts->count);
  for (int32_t i = 0; i < n; ++i) out[i] = ts->log[(ts->head + i) % ts->cap];
  if (n > 0) {
    ts->head = (ts->head + n) % ts->cap;
    ts->count -= n;
  }
  *count = n;
  return MOE_OK;
}

}  // extern "C"

// ---------------------------------------------------------------- P runner

struct moe_p_runner {
  moe_ctx_t* ctx = nullptr;
  moe_turnstile_t* ts = nullptr;
  int64_t epoch = 0;
  int32_t layers = 0, T = 0;
  std::vector<const float*> logits;
  std::vector<const void*> x;
  std::vector<float*> out;
  hipStream_t stream = nullptr;
  int64_t timeout_us = 0;
  moe_p_epoch_stats_t stats{};
  std::thread thread;

  // Host time is split into enqueueing (between waits) and waiting.
  void run() {
    double enq = 0.0, wait = 0.0;
    auto t = Clock::now();
    auto lap = [&](double& acc) {
      const auto n = Clock::now();
      acc += std::chrono::duration<double, std::micro>(n - t).count();
      t = n;
    };
    int st = moe_turnstile_wait_permit(ts, epoch, -1, timeout_us);  // P1: before any GPU work
    lap(wait);
    int l = 0;
    for (; st == MOE_OK && l < layers; ++l) {
      if ((st = moe_route(ctx, MOE_PHASE_P, logits[l], T, stream))) break;
      if ((st = moe_dispatch_layout(ctx, MOE_PHASE_P, stream))) break;
      if ((st = moe_turnstile_publish(ts, epoch, l))) break;
      lap(enq);
      st = moe_turnstile_wait_permit(ts, epoch, l, timeout_us);  // P2
      lap(wait);
      if (st) break;
      if ((st = moe_dispatch_permute(ctx, MOE_PHASE_P, x[l], stream))) break;
      if ((st = moe_expert_ffn(ctx, MOE_PHASE_P, stream))) break;
      if ((st = moe_combine(ctx, MOE_PHASE_P, out[l], stream))) break;
    }
    // TaskDone also on failure, so that D never waits for a producer that stopped.
    const int done = moe_turnstile_done(ts, epoch);
    if (st == MOE_OK) st = done;
    lap(enq);
    stats.status = st;
    stats.layers_done = l;
    stats.enqueue_us = enq;
    stats.wait_us = wait;
    stats.t_end_ns = now_ns();
  }
};

extern "C" {

int moe_p_epoch_start(moe_ctx_t* ctx, moe_turnstile_t* ts, int64_t epoch, int32_t d_enqueued, int32_t layers,
                      int32_t T, const float* const* logits, const void* const* x, float* const* out,
                      hipStream_t stream, int64_t timeout_us, moe_p_runner_t** runner) {
  if (!runner) return MOE_ERR_INVALID_ARG;
  *runner = nullptr;
  if (!ctx || !ts || !stream || layers < 1 || T < 0 || timeout_us < 1) return MOE_ERR_INVALID_ARG;
  if (!logits || !x || !out) return MOE_ERR_INVALID_ARG;
  if (T > 0)
    for (int32_t l = 0; l < layers; ++l)
      if (!logits[l] || !x[l] || !out[l]) return MOE_ERR_INVALID_ARG;
  moe_phase_view_t v;
  int st = moe_phase_view(ctx, MOE_PHASE_P, &v);
  if (st) return st;
  if (v.state != MOE_STATE_IDLE) return MOE_ERR_STATE;
  moe_p_runner* r = new (std::nothrow) moe_p_runner();
  if (!r) return MOE_ERR_OOM;
  try {
    r->logits.assign(logits, logits + layers);
    r->x.assign(x, x + layers);
    r->out.assign(out, out + layers);
  } catch (const std::bad_alloc&) {
    delete r;
    return MOE_ERR_OOM;
  }
  r->ctx = ctx;
  r->ts = ts;
  r->epoch = epoch;
  r->layers = layers;
  r->T = T;
  r->stream = stream;
  r->timeout_us = timeout_us;
  if ((st = moe_turnstile_begin(ts, epoch, d_enqueued))) {
    delete r;
    return st;
  }
  r->stats.t_begin_ns = now_ns();
  try {
    r->thread = std::thread([r] { r->run(); });
  } catch (...) {
    moe_turnstile_done(ts, epoch);
    delete r;
    return MOE_ERR_OOM;
  }
  *runner = r;
  return MOE_OK;
}

int moe_p_epoch_join(moe_p_runner_t* runner, moe_p_epoch_stats_t* stats) {
  if (!runner) return MOE_ERR_INVALID_ARG;
  if (runner->thread.joinable()) runner->thread.join();
  const int st = runner->stats.status;
  if (stats) *stats = runner->stats;
  delete runner;
  return st;
}

}  // extern "C"
