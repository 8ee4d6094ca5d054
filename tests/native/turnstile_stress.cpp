// Host-only stress driver for the segment turnstile (Sections 4.2-4.3) and
// the P-epoch runner, built from the library's own turnstile.cpp with a
// sanitizer (ThreadSanitizer, or AddressSanitizer + UndefinedBehaviorSanitizer)
// by tests/test_sanitize_turnstile.py.  The layer calls the runner makes are
// host-only stand-ins defined here (no GPU, no HIP runtime): they check the
// call order of one phase and count the layers, so the runner's thread and the
// controller are exercised exactly as in the library.
//
// Exit status 0: every protocol call returned what the protocol says, every
// epoch finished, and the logged transitions satisfy r <= p and publish <
// enter < release per round.  Any other status names the failed check.
#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <thread>
#include <vector>

#include "moepd_turnstile.h"

// ---- stand-ins for the layer calls of one context (phase P only) ----------

struct moe_ctx {
  std::atomic<int> state{MOE_STATE_IDLE};
  std::atomic<long> layers{0};
};

static int step(moe_ctx_t* c, int phase, int from, int to) {
  if (!c || phase != MOE_PHASE_P) return MOE_ERR_INVALID_ARG;
  int s = from;
  if (!c->state.compare_exchange_strong(s, to)) return MOE_ERR_STATE;
  return MOE_OK;
}

extern "C" {
int moe_route(moe_ctx_t* c, int phase, const float* logits, int32_t T, hipStream_t s) {
  (void)logits, (void)T, (void)s;
  return step(c, phase, MOE_STATE_IDLE, MOE_STATE_ROUTED);
}
int moe_dispatch_layout(moe_ctx_t* c, int phase, hipStream_t s) {
  (void)s;
  return step(c, phase, MOE_STATE_ROUTED, MOE_STATE_LAID_OUT);
}
int moe_dispatch_permute(moe_ctx_t* c, int phase, const void* x, hipStream_t s) {
  (void)x, (void)s;
  return step(c, phase, MOE_STATE_LAID_OUT, MOE_STATE_DISPATCHED);
}
int moe_expert_ffn(moe_ctx_t* c, int phase, hipStream_t s) {
  (void)s;
  return step(c, phase, MOE_STATE_DISPATCHED, MOE_STATE_COMPUTED);
}
int moe_combine(moe_ctx_t* c, int phase, void* out, hipStream_t s) {
  (void)out, (void)s;
  const int st = step(c, phase, MOE_STATE_COMPUTED, MOE_STATE_IDLE);
  if (st == MOE_OK) c->layers.fetch_add(1);
  return st;
}
int moe_phase_view(const moe_ctx_t* c, int phase, moe_phase_view_t* v) {
  if (!c || !v || phase != MOE_PHASE_P) return MOE_ERR_INVALID_ARG;
  *v = moe_phase_view_t{};
  v->state = c->state.load();
  return MOE_OK;
}
}

#define REQUIRE(cond, what)                                      \
  do {                                                           \
    if (!(cond)) {                                               \
      std::fprintf(stderr, "FAILED: %s (line %d)\n", what, __LINE__); \
      std::exit(1);                                              \
    }                                                            \
  } while (0)

// D's side: enter at each boundary the controller offers, release, until the
// epoch's task is done (then one last release).
static void d_loop(moe_turnstile_t* ts, std::atomic<bool>* stop, long* rounds) {
  while (!stop->load()) {
    const int st = moe_turnstile_wait_boundary(ts, 2000);
    if (st == MOE_ERR_TIMEOUT) continue;
    REQUIRE(st == MOE_OK, "wait_boundary");
    // (the state is not checked here: a D that passed while no epoch was
    // active may find the next epoch begun; the log check covers the order)
    moe_turnstile_state_t q;
    REQUIRE(moe_turnstile_query(ts, &q) == MOE_OK, "query");
    REQUIRE(moe_turnstile_release(ts) == MOE_OK, "release");
    ++*rounds;
  }
}

static void check_log(moe_turnstile_t* ts) {
  std::vector<moe_turnstile_event_t> ev(1 << 16);
  int32_t n = 0;
  REQUIRE(moe_turnstile_log(ts, ev.data(), (int32_t)ev.size(), &n) == MOE_OK, "log");
  int64_t r = -1, p = 0;
  bool inside = false;
  for (int32_t i = 0; i < n; ++i) {
    const auto& e = ev[i];
    switch (e.kind) {
      // (a D inside when an epoch begins stays inside: it entered while no
      // task was active and releases no permit of the new epoch)
      case MOE_TS_EV_BEGIN: r = -1; p = e.value; break;
      case MOE_TS_EV_PUBLISH: REQUIRE(e.value > r && e.value <= p, "publish within the permit"); r = e.value; break;
      case MOE_TS_EV_RESUME: REQUIRE(e.value < p, "P resumed below the permit"); break;
      case MOE_TS_EV_ENTER: REQUIRE(!inside, "D entered twice"); inside = true; break;
      case MOE_TS_EV_RELEASE: REQUIRE(inside, "release without entry"); inside = false; p = e.value; break;
      case MOE_TS_EV_DONE: break;
      default: REQUIRE(false, "unknown event kind");
    }
    REQUIRE(r <= p || e.kind == MOE_TS_EV_DONE || e.kind == MOE_TS_EV_RELEASE, "r <= p");
  }
}

int main(int argc, char** argv) {
  const int epochs = argc > 1 ? std::atoi(argv[1]) : 200;
  std::mt19937 rng(12345);

  // 1. The controller driven directly by a P thread and a D thread.
  {
    moe_turnstile_t* ts = nullptr;
    REQUIRE(moe_turnstile_create(1, 1 << 16, &ts) == MOE_OK, "create");
    std::atomic<bool> stop{false};
    long rounds = 0;
    std::thread d(d_loop, ts, &stop, &rounds);
    for (int e = 0; e < epochs; ++e) {
      REQUIRE(moe_turnstile_set_span(ts, 1 + (int)(rng() % 4)) == MOE_OK, "set_span");
      const int B = 1 + (int)(rng() % 9);
      REQUIRE(moe_turnstile_begin(ts, e, (int)(rng() & 1)) == MOE_OK, "begin");
      REQUIRE(moe_turnstile_wait_permit(ts, e, -1, 10000000) == MOE_OK, "P1 wait");
      for (int b = 0; b < B; ++b) {
        REQUIRE(moe_turnstile_publish(ts, e, b) == MOE_OK, "publish");
        REQUIRE(moe_turnstile_wait_permit(ts, e, b, 10000000) == MOE_OK, "P2 wait");
      }
      REQUIRE(moe_turnstile_done(ts, e) == MOE_OK, "done");
    }
    stop.store(true);
    d.join();
    check_log(ts);
    moe_turnstile_state_t q;
    REQUIRE(moe_turnstile_query(ts, &q) == MOE_OK && q.task == MOE_TS_DONE, "final state");
    REQUIRE(moe_turnstile_destroy(ts) == MOE_OK, "destroy");
    std::printf("controller: %d epochs, %ld D rounds\n", epochs, rounds);
  }

  // 2. The P-epoch runner's thread against a D thread, on the stand-in layer.
  {
    moe_turnstile_t* ts = nullptr;
    REQUIRE(moe_turnstile_create(2, 1 << 16, &ts) == MOE_OK, "create");
    moe_ctx ctx;
    const int L = 7;
    float lg[1];
    unsigned char xb[1];
    float ob[1];
    std::vector<const float*> logits(L, lg);
    std::vector<const void*> x(L, xb);
    std::vector<float*> out(L, ob);
    hipStream_t s = reinterpret_cast<hipStream_t>(0x1);
    std::atomic<bool> stop{false};
    long rounds = 0;
    std::thread d(d_loop, ts, &stop, &rounds);
    const int runs = epochs / 10 + 1;
    for (int e = 0; e < runs; ++e) {
      moe_p_runner_t* r = nullptr;
      REQUIRE(moe_p_epoch_start(&ctx, ts, e, (int)(rng() & 1), L, 16, logits.data(), x.data(), out.data(), s,
                                10000000, &r) == MOE_OK, "epoch start");
      moe_p_epoch_stats_t st;
      REQUIRE(moe_p_epoch_join(r, &st) == MOE_OK, "epoch join");
      REQUIRE(st.layers_done == L, "layers done");
    }
    stop.store(true);
    d.join();
    check_log(ts);
    REQUIRE(ctx.layers.load() == (long)runs * L, "stand-in layer count");
    REQUIRE(moe_turnstile_destroy(ts) == MOE_OK, "destroy");
    std::printf("runner: %d epochs of %d layers, %ld D rounds\n", runs, L, rounds);
  }
  std::printf("ok\n");
  return 0;
}
