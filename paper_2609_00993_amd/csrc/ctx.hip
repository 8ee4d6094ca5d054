// Host runtime of libmoepd: the context, the per-phase state sets and the
// C-ABI entry points declared in include/moepd.h.
//
// Phase ownership follows Section 5.1 of the paper (table "Ownership in the
// concurrent DeepEP runtime"): the weights are shared and read-only, while
// each phase owns its buffers, counters (the dispatch histogram cells and
// per-expert counts), workspace and events, selected by an explicit phase id
// (Section 5.1, Section 6).  Each phase's buffers live in one allocation made
// at creation, so their addresses never change (the D phase replays against
// fixed addresses) and the two phases' address ranges are disjoint.  A phase
// admits one pending operation at a time and moves through explicit states
// (Section 5.2); a reset is refused until the phase's enqueued work is done
// (Section 5.3).
#include <atomic>
#include <new>
#include <string.h>

#include "kernels.h"
#include "moepd.h"
#include "moepd_turnstile.h"

using namespace moepd;

namespace {

constexpr size_t kAlign = 256;

inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

struct Timing {
  hipEvent_t* start = nullptr;
  hipEvent_t* stop = nullptr;
  int capacity = 0;
  int used = 0;
};

struct Phase {
  int state = MOE_STATE_IDLE;
  int T = 0;
  int regime = 0;  // tile shape (ffn_bf16_bm / ffn_mx_bm): 0 large batch, 1 small, 2 very large (bf16)
  int bm = 0;
  int chunk_tokens = 1;
  int nchunks = 1;
  int max_tokens = 0;
  long long rows_cap = 0;
  int router_cap = 0;  // rows of the router's partial-product buffer
  PhaseBuffers b{};
  void* mem = nullptr;
  hipEvent_t ev = nullptr;
  bool ev_recorded = false;
  hipStream_t last_stream = nullptr;
  // Generation stored in the signal word while this phase's layer window is
  // open.  A reset moves to a new generation, so a window left open by an
  // abandoned layer is no longer honoured.
  int32_t gen = 1;
  // The current call's stream is being captured into a graph (set by enter).
  bool capturing = false;
  Timing timing[MOE_NUM_KERNELS];
};

}  // namespace

struct moe_ctx {
  moe_config_t cfg;
  moe_weights_t w;
  int device;
  int esz;
  Phase ph[MOE_NUM_PHASES];
  // Tile regime of each phase's latest bf16 expert-FFN launch (-1: none).
  // The other phase reads it (possibly from another host thread) to choose
  // its decode tiles: 160-row prefill tiles leave 4 KB of a CU's LDS free,
  // too little for the LDS-staged decode tile, so beside them the phase takes
  // the tile that needs no LDS and can share their CUs.  Only a performance
  // choice: both tiles give the same results.
  std::atomic<int> ffn_regime[MOE_NUM_PHASES] = {-1, -1};
};

namespace {

bool valid_config(const moe_config_t* c) {
  if (c->num_experts < 1 || c->num_experts > kMaxExperts) return false;
  if (c->num_local_experts < 1 || c->num_local_experts > kMaxLocalExperts) return false;
  if (c->expert_begin < 0 || c->expert_begin + c->num_local_experts > c->num_experts) return false;
  if (c->top_k < 1 || c->top_k > kMaxTopK || c->top_k > c->num_experts) return false;
  if (c->hidden < 64 || c->hidden > 16384 || c->hidden % 64) return false;
  if (c->inter < 64 || c->inter > 16384 || c->inter % 64) return false;
  if (c->dtype != MOE_DTYPE_F32 && c->dtype != MOE_DTYPE_BF16 && c->dtype != MOE_DTYPE_FP8) return false;
  // MX FP8 GEMMs step through K 128 values at a time
  if (c->dtype == MOE_DTYPE_FP8 && (c->hidden % 128 || c->inter % 128)) return false;
  for (int p = 0; p < MOE_NUM_PHASES; ++p)
    if (c->max_tokens[p] < 0 || c->max_tokens[p] > (1 << 20)) return false;
  if (c->flags != 0) return false;
  if (c->d_priority_us < 0 || c->d_priority_us > 1000) return false;
  return true;
}

int max_chunks(int e_loc) { return kMaxCells / e_loc; }

void free_timing(Phase& p) {
  for (int k = 0; k < MOE_NUM_KERNELS; ++k) {
    Timing& t = p.timing[k];
    for (int i = 0; i < t.capacity; ++i) {
      if (t.start && t.start[i]) (void)hipEventDestroy(t.start[i]);
      if (t.stop && t.stop[i]) (void)hipEventDestroy(t.stop[i]);
    }
    delete[] t.start;
    delete[] t.stop;
    t = Timing{};
  }
}

void free_phase(Phase& p) {
  free_timing(p);
  if (p.ev) (void)hipEventDestroy(p.ev);
  if (p.mem) (void)hipFree(p.mem);
  p.ev = nullptr;
  p.mem = nullptr;
}

int alloc_phase(moe_ctx* ctx, int phase) {
  const moe_config_t& c = ctx->cfg;
  Phase& p = ctx->ph[phase];
  p.max_tokens = c.max_tokens[phase];
  const long long slots = (long long)p.max_tokens * c.top_k;
  const int kk = c.top_k < c.num_local_experts ? c.top_k : c.num_local_experts;
  p.rows_cap = (long long)p.max_tokens * kk;
  const int E = c.num_local_experts;
  const int mc = max_chunks(E);

  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes > 0 ? bytes : 1);
    return o;
  };
  const size_t o_idx = take(slots * 4), o_w = take(slots * 4), o_cnt = take(E * 4), o_off = take((E + 1) * 4);
  const size_t o_ros = take(slots * 4), o_tor = take(p.rows_cap * 4);
  const size_t o_xp = take(p.rows_cap * c.hidden * ctx->esz), o_h = take(p.rows_cap * c.inter * ctx->esz);
  const size_t o_y = take(p.rows_cap * c.hidden * 4);
  // Router GEMM: the logits, and room for its K-split partial products (at
  // least 4096 rows, so that small batches can split K many ways).
  p.router_cap = c.dtype != MOE_DTYPE_F32 ? (p.max_tokens > 4096 ? p.max_tokens : 4096) : 0;
  const size_t o_lg = take((size_t)p.max_tokens * c.num_experts * 4);
  const size_t o_part = take((size_t)p.router_cap * c.num_experts * 4);
  // The signal slot is 16 bytes: the grouped GEMMs read the window word in it
  // with a 16-byte LDS DMA (its other words stay zero).
  const size_t o_cc = take((size_t)E * mc * 4), o_tb = take((E + 1) * 4), o_sig = take(16);
  const size_t o_td = take(c.dtype == MOE_DTYPE_BF16 ? (size_t)ffn_bf16_handover_words(p.rows_cap, E, c.hidden) * 4 : 0);

  void* mem = nullptr;
  if (hipMalloc(&mem, off) != hipSuccess || !mem) {
    (void)hipGetLastError();
    return MOE_ERR_OOM;
  }
  p.mem = mem;
  char* base = (char*)mem;
  p.b.topk_idx = (int32_t*)(base + o_idx);
  p.b.topk_w = (float*)(base + o_w);
  p.b.counts = (int32_t*)(base + o_cnt);
  p.b.offsets = (int32_t*)(base + o_off);
  p.b.row_of_slot = (int32_t*)(base + o_ros);
  p.b.token_of_row = (int32_t*)(base + o_tor);
  p.b.x_perm = base + o_xp;
  p.b.h = base + o_h;
  p.b.y = (float*)(base + o_y);
  p.b.chunk_counts = (int32_t*)(base + o_cc);
  p.b.tile_base = (int32_t*)(base + o_tb);
  p.b.signal = (int32_t*)(base + o_sig);
  p.b.tile_done = (int32_t*)(base + o_td);
  p.b.logits = (float*)(base + o_lg);
  p.b.partials = (float*)(base + o_part);
  // Zero the small metadata (counts, offsets, tile prefix, signal word, tile
  // marks) once at creation.
  if (hipMemset(base + o_cnt, 0, o_ros - o_cnt) != hipSuccess) return MOE_ERR_HIP;
  if (hipMemset(base + o_tb, 0, off - o_tb) != hipSuccess) return MOE_ERR_HIP;
  if (hipEventCreateWithFlags(&p.ev, hipEventDisableTiming) != hipSuccess) {
    p.ev = nullptr;
    return MOE_ERR_HIP;
  }
  return MOE_OK;
}

inline int check_phase(const moe_ctx* ctx, int phase) {
  if (!ctx) return MOE_ERR_INVALID_ARG;
  if (phase != MOE_PHASE_P && phase != MOE_PHASE_D) return MOE_ERR_INVALID_PHASE;
  return MOE_OK;
}

// Order this phase's next work after its previous work when the stream changes.
// Stream hand-over and graph capture.  A phase driven on a new stream makes
// that stream wait for the phase's last recorded event.  While `s` is being
// captured into a graph (a D layer captured once and replayed, Section 6.1),
// the captured kernels are ordered by the stream itself: no event is
// recorded or waited on and no timing events are taken, and a hand-over
// from another stream into a capture is refused (the wait could not be
// part of the graph): run the phase on the capturing stream first.
int enter(moe_ctx* ctx, Phase& p, hipStream_t s) {
  if (hipSetDevice(ctx->device) != hipSuccess) return MOE_ERR_HIP;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cs) != hipSuccess) return MOE_ERR_HIP;
  p.capturing = cs != hipStreamCaptureStatusNone;
  if (p.ev_recorded && p.last_stream != s) {
    if (p.capturing) return MOE_ERR_STATE;
    if (hipStreamWaitEvent(s, p.ev, 0) != hipSuccess) return MOE_ERR_HIP;
  }
  return MOE_OK;
}

int leave(Phase& p, hipStream_t s) {
  if (!p.capturing) {
    if (hipEventRecord(p.ev, s) != hipSuccess) return MOE_ERR_HIP;
    p.ev_recorded = true;
  }
  p.last_stream = s;
  return MOE_OK;
}

// Launch wrapper: brackets the launch with timing events when enabled.
template <typename F>
int timed(Phase& p, int kernel, hipStream_t s, F&& launch) {
  Timing& t = p.timing[kernel];
  const bool rec = !p.capturing && t.capacity > 0 && t.used < t.capacity;
  if (rec && hipEventRecord(t.start[t.used], s) != hipSuccess) return MOE_ERR_HIP;
  if (launch() != hipSuccess) return MOE_ERR_HIP;
  if (rec) {
    if (hipEventRecord(t.stop[t.used], s) != hipSuccess) return MOE_ERR_HIP;
    ++t.used;
  }
  return MOE_OK;
}

// The D phase announces its layer window when D-first admission is on.
WindowSignal window_of(moe_ctx* ctx, int phase) {
  if (phase != MOE_PHASE_D || ctx->cfg.d_priority_us <= 0) return WindowSignal{nullptr, 0};
  Phase& p = ctx->ph[phase];
  return WindowSignal{p.b.signal, p.gen};
}

// The P phase's grouped GEMMs hold back while the D window is open; one poll
// sleeps 127 * 64 cycles, about 3.4 us at 2.4 GHz.  Not for tiles whose
// workgroups hold too many registers for a D GEMM wave to share their SIMDs
// (the bf16 256-row tiles, 460 VGPRs; the MX FP8 ring tiles, 476-480): a P
// workgroup waiting on its CU would only keep D off it.
YieldTo yield_of(moe_ctx* ctx, int phase) {
  if (phase != MOE_PHASE_P || ctx->cfg.d_priority_us <= 0) return YieldTo{nullptr, 0, 0};
  const int regime = ctx->ph[phase].regime;
  if (regime == 2 || (ctx->cfg.dtype == MOE_DTYPE_FP8 && regime == 0)) return YieldTo{nullptr, 0, 0};
  const Phase& d = ctx->ph[MOE_PHASE_D];
  return YieldTo{d.b.signal, d.gen, (ctx->cfg.d_priority_us * 10 + 33) / 34};
}
// MX FP8 contexts keep E4M3 codes and their scale bytes in the x_perm and h
// regions (sized for bf16 rows, so codes plus scales fit).
MxBuffers mx_of(const moe_ctx* ctx, const Phase& p) {
  const size_t R = (size_t)p.rows_cap;
  uint8_t* xp = static_cast<uint8_t*>(p.b.x_perm);
  uint8_t* h = static_cast<uint8_t*>(p.b.h);
  return MxBuffers{xp, xp + R * ctx->cfg.hidden, h, h + R * ctx->cfg.inter};
}

// Dispatch notification (Section 5.2): the per-chunk histogram, then the
// prefix sum and stable row assignment.  Picks the phase's tile regime.
int layout(moe_ctx* ctx, Phase& p, hipStream_t stream) {
  const moe_config_t& c = ctx->cfg;
  const int T = p.T, k = c.top_k, E_loc = c.num_local_experts;
  dispatch_chunking(T, k, E_loc, &p.chunk_tokens, &p.nchunks);
  if (c.dtype == MOE_DTYPE_FP8) {
    const long long avg = (long long)T * k / c.num_experts;
    p.regime = avg >= 32 ? 0 : 1;
    p.bm = ffn_mx_bm(p.regime);
  } else if (c.dtype == MOE_DTYPE_BF16) {
    // Rows per resident expert expected under even routing: T*k/E.  Small
    // batches stream weights (32-row tiles); large ones take 160-row tiles,
    // and very large ones 256-row tiles, which move fewer bytes into LDS per
    // flop.
    const long long avg = (long long)T * k / c.num_experts;
    p.regime = avg >= 512 ? 2 : avg >= 32 ? 0 : 1;
    p.bm = ffn_bf16_bm(p.regime);
  } else {
    p.regime = 0;
    p.bm = ffn_f32_bm();
  }
  int st = MOE_OK;
  if (p.nchunks > 1) {  // one chunk: the place kernel counts its slots itself
    st = timed(p, MOE_KERNEL_COUNT, stream, [&] {
      return launch_count(p.b.topk_idx, T, k, c.expert_begin, E_loc, p.chunk_tokens, p.nchunks, p.b, stream);
    });
    if (st) return st;
  }
  return timed(p, MOE_KERNEL_PLACE, stream, [&] {
    return launch_place(p.b.topk_idx, T, k, c.expert_begin, E_loc, p.chunk_tokens, p.nchunks, p.bm, p.b, stream);
  });
}

// Dispatch data movement: token rows into expert-contiguous rows.
int permute(moe_ctx* ctx, Phase& p, const void* x, hipStream_t stream) {
  if (p.T == 0) return MOE_OK;
  if (ctx->cfg.dtype == MOE_DTYPE_FP8) {
    const MxBuffers mx = mx_of(ctx, p);
    return timed(p, MOE_KERNEL_PERMUTE, stream, [&] {
      return launch_permute_mx(x, p.T, ctx->cfg.top_k, ctx->cfg.hidden, p.b.row_of_slot, mx.x_codes, mx.x_scales,
                               stream);
    });
  }
  return timed(p, MOE_KERNEL_PERMUTE, stream, [&] {
    return launch_permute(x, p.T, ctx->cfg.top_k, ctx->cfg.hidden * ctx->esz, p.b.row_of_slot, p.b.x_perm, stream);
  });
}
}  // namespace

extern "C" {

int moe_ctx_create(const moe_config_t* cfg, const moe_weights_t* w, moe_ctx_t** out) {
  if (!out) return MOE_ERR_INVALID_ARG;
  *out = nullptr;
  if (!cfg || !w || !w->w_gate_up || !w->w_down) return MOE_ERR_INVALID_ARG;
  if (!valid_config(cfg)) return MOE_ERR_INVALID_ARG;
  if (cfg->dtype == MOE_DTYPE_FP8 && (!w->w_gate_up_scales || !w->w_down_scales)) return MOE_ERR_INVALID_ARG;
  moe_ctx* ctx = new (std::nothrow) moe_ctx();
  if (!ctx) return MOE_ERR_OOM;
  ctx->cfg = *cfg;
  ctx->w = *w;
  // bytes of an x element: FP8 contexts take bf16 hidden states
  ctx->esz = cfg->dtype == MOE_DTYPE_F32 ? 4 : 2;
  if (hipGetDevice(&ctx->device) != hipSuccess) {
    delete ctx;
    return MOE_ERR_HIP;
  }
  for (int p = 0; p < MOE_NUM_PHASES; ++p) {
    const int st = alloc_phase(ctx, p);
    if (st != MOE_OK) {
      for (int q = 0; q <= p; ++q) free_phase(ctx->ph[q]);
      delete ctx;
      return st;
    }
  }
  *out = ctx;
  return MOE_OK;
}

int moe_route(moe_ctx_t* ctx, int phase, const float* logits, int32_t T, hipStream_t stream) {
  int st = check_phase(ctx, phase);
  if (st) return st;
  if (T < 0 || (T > 0 && !logits) || !stream) return MOE_ERR_INVALID_ARG;
  Phase& p = ctx->ph[phase];
  if (p.state != MOE_STATE_IDLE) return MOE_ERR_STATE;
  if (T > p.max_tokens) return MOE_ERR_CAPACITY;
  if ((st = enter(ctx, p, stream))) return st;
  const moe_config_t& c = ctx->cfg;
  if (T > 0) {
    st = timed(p, MOE_KERNEL_ROUTE, stream,
               [&] {
                 return launch_route(logits, T, c.num_experts, c.top_k, p.b.topk_idx, p.b.topk_w,
                                     window_of(ctx, phase), RouterSum{nullptr, nullptr, 1}, stream);
               });
    if (st) return st;
  }
  if ((st = leave(p, stream))) return st;
  p.T = T;
  p.state = MOE_STATE_ROUTED;
  return MOE_OK;
}

int moe_route_from_hidden(moe_ctx_t* ctx, int phase, const void* x, const void* w_router, const float* bias,
                          int32_t T, hipStream_t stream) {
  int st = check_phase(ctx, phase);
  if (st) return st;
  if (T < 0 || (T > 0 && (!x || !w_router)) || !stream) return MOE_ERR_INVALID_ARG;
  Phase& p = ctx->ph[phase];
  if (p.state != MOE_STATE_IDLE) return MOE_ERR_STATE;
  if (T > p.max_tokens) return MOE_ERR_CAPACITY;
  if ((st = enter(ctx, p, stream))) return st;
  const moe_config_t& c = ctx->cfg;
  if (T > 0) {
    int nsplit = 1;
    if (c.dtype != MOE_DTYPE_F32) {
      int ks = 0;
      nsplit = router_splits(T, c.num_experts, c.hidden, p.router_cap, &ks);
      float* dst = nsplit > 1 ? p.b.partials : p.b.logits;
      st = timed(p, MOE_KERNEL_ROUTER, stream, [&] {
        return launch_router_bf16(x, w_router, T, c.num_experts, c.hidden, dst, nsplit, ks, yield_of(ctx, phase),
                                  stream);
      });
    } else {
      st = timed(p, MOE_KERNEL_ROUTER, stream, [&] {
        return launch_router_f32((const float*)x, (const float*)w_router, T, c.num_experts, c.hidden, p.b.logits,
                                 stream);
      });
    }
    if (st) return st;
    const float* in = nsplit > 1 ? p.b.partials : p.b.logits;
    st = timed(p, MOE_KERNEL_ROUTE, stream, [&] {
      return launch_route(in, T, c.num_experts, c.top_k, p.b.topk_idx, p.b.topk_w, window_of(ctx, phase),
                          RouterSum{p.b.logits, bias, nsplit}, stream);
    });
    if (st) return st;
  }
  if ((st = leave(p, stream))) return st;
  p.T = T;
  p.state = MOE_STATE_ROUTED;
  return MOE_OK;
}

int moe_dispatch_layout(moe_ctx_t* ctx, int phase, hipStream_t stream) {
  int st = check_phase(ctx, phase);
  if (st) return st;
  Phase& p = ctx->ph[phase];
  if (!stream) return MOE_ERR_INVALID_ARG;
  if (p.state != MOE_STATE_ROUTED) return MOE_ERR_STATE;
  if ((st = enter(ctx, p, stream))) return st;
  if ((st = layout(ctx, p, stream))) return st;
  if ((st = leave(p, stream))) return st;
  p.state = MOE_STATE_LAID_OUT;
  return MOE_OK;
}

int moe_dispatch_permute(moe_ctx_t* ctx, int phase, const void* x, hipStream_t stream) {
  int st = check_phase(ctx, phase);
  if (st) return st;
  Phase& p = ctx->ph[phase];
  if (!stream) return MOE_ERR_INVALID_ARG;
  if (p.state != MOE_STATE_LAID_OUT) return MOE_ERR_STATE;
  if (p.T > 0 && !x) return MOE_ERR_INVALID_ARG;
  if ((st = enter(ctx, p, stream))) return st;
  if ((st = permute(ctx, p, x, stream))) return st;
  if ((st = leave(p, stream))) return st;
  p.state = MOE_STATE_DISPATCHED;
  return MOE_OK;
}

int moe_dispatch(moe_ctx_t* ctx, int phase, const void* x, hipStream_t stream) {
  int st = check_phase(ctx, phase);
  if (st) return st;
  Phase& p = ctx->ph[phase];
  if (!stream) return MOE_ERR_INVALID_ARG;
  if (p.state != MOE_STATE_ROUTED) return MOE_ERR_STATE;
  if (p.T > 0 && !x) return MOE_ERR_INVALID_ARG;
  if ((st = enter(ctx, p, stream))) return st;
  if ((st = layout(ctx, p, stream))) return st;
  if ((st = permute(ctx, p, x, stream))) return st;
  if ((st = leave(p, stream))) return st;
  p.state = MOE_STATE_DISPATCHED;
  return MOE_OK;
}

int moe_expert_ffn(moe_ctx_t* ctx, int phase, hipStream_t stream) {
  int st = check_phase(ctx, phase);
  if (st) return st;
  Phase& p = ctx->ph[phase];
  if (!stream) return MOE_ERR_INVALID_ARG;
  if (p.state != MOE_STATE_DISPATCHED) return MOE_ERR_STATE;
  if ((st = enter(ctx, p, stream))) return st;
  const moe_config_t& c = ctx->cfg;
  if (p.T > 0) {
    const int kk = c.top_k < c.num_local_experts ? c.top_k : c.num_local_experts;
    const long long rows = (long long)p.T * kk;
    const int max_m_tiles = (int)((rows + p.bm - 1) / p.bm) + c.num_local_experts;
    ctx->ffn_regime[phase].store(p.regime, std::memory_order_relaxed);
    const int other = ctx->ffn_regime[phase ^ 1].load(std::memory_order_relaxed);
    const bool stage = other != 0;
    // D first (Section 3.1) on one GPU: while D-first admission is on and the
    // context runs D layers, P's 256-row GEMM2 takes the tile that leaves a CU
    // room for D's decode tiles beside it.
    const bool share = phase == MOE_PHASE_P && c.d_priority_us > 0 && other != -1;
    for (int gemm = 1; gemm <= 2; ++gemm) {
      st = timed(p, gemm == 1 ? MOE_KERNEL_GEMM1 : MOE_KERNEL_GEMM2, stream, [&] {
        if (c.dtype == MOE_DTYPE_FP8)
          return launch_ffn_mx(p.regime, gemm, p.b, mx_of(ctx, p),
                               MxWeights{ctx->w.w_gate_up, ctx->w.w_gate_up_scales, ctx->w.w_down, ctx->w.w_down_scales},
                               c.num_local_experts, c.hidden, c.inter, max_m_tiles, yield_of(ctx, phase), stream);
        if (c.dtype == MOE_DTYPE_BF16)
          return launch_ffn_bf16(p.regime, gemm, p.b, ctx->w.w_gate_up, ctx->w.w_down, c.num_local_experts, c.hidden,
                                 c.inter, max_m_tiles, stage, share, yield_of(ctx, phase),
                                 ctx->ph[phase ^ 1].b.signal, stream);
        return launch_ffn_f32(gemm, p.b, ctx->w.w_gate_up, ctx->w.w_down, c.num_local_experts, c.hidden, c.inter,
                              max_m_tiles, stream);
      });
      if (st) return st;
    }
  }
  if ((st = leave(p, stream))) return st;
  p.state = MOE_STATE_COMPUTED;
  return MOE_OK;
}

int moe_combine(moe_ctx_t* ctx, int phase, void* out, hipStream_t stream) {
  int st = check_phase(ctx, phase);
  if (st) return st;
  Phase& p = ctx->ph[phase];
  if (!stream) return MOE_ERR_INVALID_ARG;
  if (p.state != MOE_STATE_COMPUTED) return MOE_ERR_STATE;
  if (p.T > 0 && !out) return MOE_ERR_INVALID_ARG;
  if ((st = enter(ctx, p, stream))) return st;
  const moe_config_t& c = ctx->cfg;
  if (p.T > 0) {
    st = timed(p, MOE_KERNEL_COMBINE, stream, [&] {
      return launch_combine(p.b.y, p.b.topk_w, p.b.row_of_slot, p.T, c.top_k, c.hidden, out, window_of(ctx, phase),
                            stream);
    });
    if (st) return st;
  }
  if ((st = leave(p, stream))) return st;
  p.state = MOE_STATE_IDLE;
  return MOE_OK;
}

int moe_phase_view(const moe_ctx_t* ctx, int phase, moe_phase_view_t* v) {
  int st = check_phase(ctx, phase);
  if (st) return st;
  if (!v) return MOE_ERR_INVALID_ARG;
  const Phase& p = ctx->ph[phase];
  memset(v, 0, sizeof(*v));
  v->state = p.state;
  v->tokens = p.T;
  v->rows_capacity = (int32_t)p.rows_cap;
  v->topk_idx = p.b.topk_idx;
  v->topk_w = p.b.topk_w;
  v->counts = p.b.counts;
  v->offsets = p.b.offsets;
  v->row_of_slot = p.b.row_of_slot;
  v->token_of_row = p.b.token_of_row;
  v->x_perm = p.b.x_perm;
  v->h = p.b.h;
  v->y = p.b.y;
  v->logits = p.b.logits;
  if (ctx->cfg.dtype == MOE_DTYPE_FP8) {
    const MxBuffers mx = mx_of(ctx, p);
    v->x_perm_scales = mx.x_scales;
    v->h_scales = mx.h_scales;
  }
  return MOE_OK;
}

int moe_phase_reset(moe_ctx_t* ctx, int phase) {
  int st = check_phase(ctx, phase);
  if (st) return st;
  Phase& p = ctx->ph[phase];
  if (p.ev_recorded) {
    if (hipSetDevice(ctx->device) != hipSuccess) return MOE_ERR_HIP;
    const hipError_t q = hipEventQuery(p.ev);
    if (q == hipErrorNotReady) return MOE_ERR_BUSY;
    if (q != hipSuccess) return MOE_ERR_HIP;
  }
  p.state = MOE_STATE_IDLE;
  p.T = 0;
  p.gen = p.gen == 0x3fffffff ? 1 : p.gen + 1;
  return MOE_OK;
}

int moe_ctx_destroy(moe_ctx_t* ctx) {
  if (!ctx) return MOE_OK;
  int st = MOE_OK;
  if (hipSetDevice(ctx->device) != hipSuccess) st = MOE_ERR_HIP;
  for (int p = 0; p < MOE_NUM_PHASES; ++p) {
    if (ctx->ph[p].ev_recorded && hipEventSynchronize(ctx->ph[p].ev) != hipSuccess) st = MOE_ERR_HIP;
  }
  for (int p = 0; p < MOE_NUM_PHASES; ++p) free_phase(ctx->ph[p]);
  delete ctx;
  return st;
}

const char* moe_status_string(int status) {
  switch (status) {
    case MOE_OK: return "ok";
    case MOE_ERR_INVALID_ARG: return "invalid argument";
    case MOE_ERR_INVALID_PHASE: return "invalid phase id";
    case MOE_ERR_CAPACITY: return "batch exceeds the phase capacity";
    case MOE_ERR_STATE: return "call out of order for the phase state";
    case MOE_ERR_BUSY: return "phase has work in flight";
    case MOE_ERR_OOM: return "device allocation failed";
    case MOE_ERR_HIP: return "HIP runtime error";
    case MOE_ERR_REJECTED: return "turnstile refused the call";
    case MOE_ERR_TIMEOUT: return "turnstile wait timed out";
    default: return "unknown status";
  }
}

int moe_timing_enable(moe_ctx_t* ctx, int32_t max_launches) {
  if (!ctx || max_launches < 0 || max_launches > (1 << 16)) return MOE_ERR_INVALID_ARG;
  if (hipSetDevice(ctx->device) != hipSuccess) return MOE_ERR_HIP;
  for (int ph = 0; ph < MOE_NUM_PHASES; ++ph) {
    Phase& p = ctx->ph[ph];
    if (p.ev_recorded) {
      const hipError_t q = hipEventQuery(p.ev);
      if (q == hipErrorNotReady) return MOE_ERR_BUSY;
      if (q != hipSuccess) return MOE_ERR_HIP;
    }
  }
  for (int ph = 0; ph < MOE_NUM_PHASES; ++ph) {
    Phase& p = ctx->ph[ph];
    free_timing(p);
    if (max_launches == 0) continue;
    for (int k = 0; k < MOE_NUM_KERNELS; ++k) {
      Timing& t = p.timing[k];
      t.start = new (std::nothrow) hipEvent_t[max_launches]();
      t.stop = new (std::nothrow) hipEvent_t[max_launches]();
      if (!t.start || !t.stop) {
        free_timing(p);
        return MOE_ERR_OOM;
      }
      t.capacity = max_launches;
      for (int i = 0; i < max_launches; ++i) {
        if (hipEventCreate(&t.start[i]) != hipSuccess || hipEventCreate(&t.stop[i]) != hipSuccess) {
          free_timing(p);
          return MOE_ERR_HIP;
        }
      }
    }
  }
  return MOE_OK;
}

int moe_timing_read(moe_ctx_t* ctx, int phase, int kernel, double* total_ms, int32_t* launches) {
  int st = check_phase(ctx, phase);
  if (st) return st;
  if (kernel < 0 || kernel >= MOE_NUM_KERNELS || !total_ms || !launches) return MOE_ERR_INVALID_ARG;
  if (hipSetDevice(ctx->device) != hipSuccess) return MOE_ERR_HIP;
  Timing& t = ctx->ph[phase].timing[kernel];
  double sum = 0.0;
  for (int i = 0; i < t.used; ++i) {
    float ms = 0.f;
    if (hipEventSynchronize(t.stop[i]) != hipSuccess) return MOE_ERR_HIP;
    if (hipEventElapsedTime(&ms, t.start[i], t.stop[i]) != hipSuccess) return MOE_ERR_HIP;
    sum += ms;
  }
  *total_ms = sum;
  *launches = t.used;
  t.used = 0;
  return MOE_OK;
}

const char* moe_kernel_name(int kernel) {
  static const char* names[MOE_NUM_KERNELS] = {"route", "count",   "place",      "permute",
                                               "gemm1_swiglu", "gemm2_down", "combine", "router_gemm"};
  return (kernel >= 0 && kernel < MOE_NUM_KERNELS) ? names[kernel] : "?";
}

}  // extern "C"
