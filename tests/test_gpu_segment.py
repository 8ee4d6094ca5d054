"""GPU: dispatch split at its notification boundary (Section 5.2) and the
P-epoch runner driven through the segment turnstile (Sections 4.2-4.3).

Segmenting P changes only when its work is enqueued, never what it computes:
the split dispatch enqueues the same kernels as moe_dispatch, and a P epoch
run through the turnstile with D iterations let in at its boundaries gives
every layer's output bit for bit as the same layers run back to back (and D
its solo output).  The order of the host transitions is checked against the
protocol model.  Failure paths are forced from the host (a batch above the
phase's capacity, a permit that never comes): every kernel still ends
normally."""

import time

import numpy as np
import pytest

import oracle
from oracle import turnstile as O
from synth import BF16, LayerSpec, make_layer
from tests.gpu_util import GpuLayer, assert_close_rms, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


SPEC = LayerSpec("seg-bf16", E=16, e0=4, E_loc=8, k=2, H=256, I=256, dtype=BF16, T_P=600, T_D=4)
LAYERS = 5


@pytest.fixture(scope="module")
def setup():
    import torch

    base = make_layer(SPEC, seed=21)
    g = GpuLayer(base)
    per = [make_layer(SPEC, seed=30 + l) for l in range(LAYERS)]
    xs = [to_dev(p.x_bits[0]) for p in per]
    lg = [to_dev(p.logits[0]) for p in per]
    M = g.M
    # Buffers are filled on torch's current stream, which our streams do not
    # wait for: synchronize before any of our work writes them.
    solo = [torch.zeros((SPEC.T_P, SPEC.H), dtype=torch.float32, device="cuda") for _ in range(LAYERS)]
    torch.cuda.synchronize()
    for l in range(LAYERS):
        M.layer(g.ctx, 0, lg[l], SPEC.T_P, xs[l], solo[l], g.streams[0])
    g.run(1)
    torch.cuda.synchronize()
    d_ref = g.out[1].clone()
    # the oracle's outputs of every P layer (each layer's own hidden rows and
    # logits, the context's weights) and of the D batch
    global ORACLE_P, ORACLE_D
    ORACLE_P = [oracle.layer(p.logits[0], p.x[0], base.w_gu, base.w_dn, SPEC.k, SPEC.e0)["out"] for p in per]
    ORACLE_D = oracle.layer(base.logits[1], base.x[1], base.w_gu, base.w_dn, SPEC.k, SPEC.e0)["out"]
    for l in range(LAYERS):
        assert_close_rms(solo[l].cpu().numpy(), ORACLE_P[l], TOL, f"P layer {l} back to back")
    assert_close_rms(d_ref.cpu().numpy(), ORACLE_D, TOL, "D layer")
    yield g, xs, lg, solo, d_ref
    g.close()


TOL = 2e-2  # bf16 layers: max|err| <= 2e-2 x RMS of the oracle's output
ORACLE_P, ORACLE_D = None, None


def _events(M, ts):
    kind = {M.MOE_TS_EV_BEGIN: "begin", M.MOE_TS_EV_PUBLISH: "publish", M.MOE_TS_EV_RESUME: "resume",
            M.MOE_TS_EV_ENTER: "enter", M.MOE_TS_EV_RELEASE: "release", M.MOE_TS_EV_DONE: "done"}
    st, ev = M.moe_turnstile_log(ts, 4096)
    M.check(st)
    return [(kind[k], e, v) for k, e, v, _ in ev]


def test_split_dispatch_matches_fused(setup):
    import torch

    g, xs, lg, solo, _ = setup
    M, ctx, s = g.M, g.ctx, g.streams[0]
    T = SPEC.T_P
    assert M.moe_dispatch_permute(ctx, 0, xs[0], s) == M.MOE_ERR_STATE  # IDLE
    M.check(M.moe_route(ctx, 0, lg[0], T, s))
    assert M.moe_dispatch_permute(ctx, 0, xs[0], s) == M.MOE_ERR_STATE  # ROUTED: layout first
    M.check(M.moe_dispatch_layout(ctx, 0, s))
    assert M.moe_phase_view(ctx, 0)[1].state == M.MOE_STATE_LAID_OUT
    assert M.moe_dispatch_layout(ctx, 0, s) == M.MOE_ERR_STATE
    assert M.moe_dispatch(ctx, 0, xs[0], s) == M.MOE_ERR_STATE
    assert M.moe_expert_ffn(ctx, 0, s) == M.MOE_ERR_STATE
    assert M.moe_dispatch_permute(ctx, 0, None, s) == M.MOE_ERR_INVALID_ARG
    M.check(M.moe_dispatch_permute(ctx, 0, xs[0], s))
    M.check(M.moe_expert_ffn(ctx, 0, s))
    out = torch.zeros_like(solo[0])
    torch.cuda.synchronize()
    M.check(M.moe_combine(ctx, 0, out, s))
    torch.cuda.synchronize()
    assert torch.equal(out, solo[0])
    # cancellation from the boundary: reset once the layout has drained
    M.check(M.moe_route(ctx, 0, lg[1], T, s))
    M.check(M.moe_dispatch_layout(ctx, 0, s))
    torch.cuda.synchronize()
    M.check(M.moe_phase_reset(ctx, 0))
    assert M.moe_phase_view(ctx, 0)[1].state == M.MOE_STATE_IDLE
    M.layer(ctx, 0, lg[1], T, xs[1], out, s)
    torch.cuda.synchronize()
    assert torch.equal(out, solo[1])


@pytest.mark.parametrize("K,d_enqueued", [(1, True), (2, True), (2, False), (8, True)])
def test_segmented_epoch_matches_back_to_back(setup, K, d_enqueued):
    import torch

    g, xs, lg, solo, d_ref = setup
    M, ctx = g.M, g.ctx
    print(f"[segment] K={K} d_enqueued={d_enqueued} layers={LAYERS}", flush=True)
    outs = [torch.full_like(solo[0], float("nan")) for _ in range(LAYERS)]
    d_bufs = [torch.zeros_like(d_ref) for _ in range(LAYERS + 2)]
    torch.cuda.synchronize()
    st, ts = M.moe_turnstile_create(K, 4096)
    M.check(st)
    d_outs = []
    try:
        st, runner = M.moe_p_epoch_start(ctx, ts, 0, d_enqueued, SPEC.T_P, lg, xs, outs, g.streams[0], 20_000_000)
        M.check(st, "moe_p_epoch_start")
        try:
            while True:
                M.check(M.moe_turnstile_wait_boundary(ts, 20_000_000), "wait_boundary")
                q = M.moe_turnstile_query(ts)[1]
                if q.task == M.MOE_TS_DONE:
                    M.check(M.moe_turnstile_release(ts))
                    break
                o = d_bufs[len(d_outs)]
                M.layer(ctx, 1, g.logits[1], SPEC.T_D, g.x[1], o, g.streams[1])
                d_outs.append(o)
                M.check(M.moe_turnstile_release(ts))
        finally:
            st, stats = M.moe_p_epoch_join(runner)
        M.check(st, "p epoch")
        assert stats.layers_done == LAYERS and stats.status == M.MOE_OK
        q = M.moe_turnstile_query(ts)[1]
        assert q.rounds == O.interior_stops(LAYERS, K) + (0 if d_enqueued else 1)
        assert len(d_outs) == q.rounds
        assert O.check_log(_events(M, ts), K) == []
    finally:
        M.moe_turnstile_destroy(ts)
    torch.cuda.synchronize()
    for l in range(LAYERS):
        assert torch.equal(outs[l], solo[l]), f"layer {l}"
        assert_close_rms(outs[l].cpu().numpy(), ORACLE_P[l], TOL, f"segmented P layer {l}")
    for i, o in enumerate(d_outs):
        assert torch.equal(o, d_ref)
        assert_close_rms(o.cpu().numpy(), ORACLE_D, TOL, f"D layer let in at boundary {i}")
    assert M.moe_phase_view(ctx, 0)[1].state == M.MOE_STATE_IDLE


def test_ready_d_runs_before_p_touches_the_gpu(setup):
    import torch

    g, xs, lg, solo, _ = setup
    M, ctx = g.M, g.ctx
    outs = [torch.zeros_like(solo[0]) for _ in range(LAYERS)]
    torch.cuda.synchronize()
    st, ts = M.moe_turnstile_create(LAYERS, 256)
    M.check(st)
    try:
        st, runner = M.moe_p_epoch_start(ctx, ts, 7, False, SPEC.T_P, lg, xs, outs, g.streams[0], 20_000_000)
        M.check(st)
        time.sleep(0.05)
        q = M.moe_turnstile_query(ts)[1]
        assert q.permit == 0 and q.reached == -1
        assert M.moe_phase_view(ctx, 0)[1].state == M.MOE_STATE_IDLE  # nothing enqueued
        M.check(M.moe_turnstile_wait_boundary(ts, 0))  # p = 0: no publication needed
        M.check(M.moe_turnstile_release(ts))
        st, stats = M.moe_p_epoch_join(runner)
        M.check(st)
        assert stats.wait_us > 40_000
    finally:
        M.moe_turnstile_destroy(ts)
    torch.cuda.synchronize()
    for l in range(LAYERS):
        assert torch.equal(outs[l], solo[l])


def test_failing_epoch_reports_taskdone(setup):
    g, xs, lg, solo, _ = setup
    M, ctx = g.M, g.ctx
    st, ts = M.moe_turnstile_create(2, 0)
    M.check(st)
    try:
        # a batch above the phase's capacity: moe_route refuses it on the host
        st, runner = M.moe_p_epoch_start(ctx, ts, 0, True, SPEC.T_P + 1, lg, xs, solo, g.streams[0], 5_000_000)
        M.check(st)
        st, stats = M.moe_p_epoch_join(runner)
        assert st == M.MOE_ERR_CAPACITY and stats.layers_done == 0
        assert M.moe_turnstile_query(ts)[1].task == M.MOE_TS_DONE
        M.check(M.moe_turnstile_wait_boundary(ts, 0))  # D is not held by a stopped producer
        M.check(M.moe_turnstile_release(ts))
        # a permit that never comes: the wait before the GPU times out
        st, runner = M.moe_p_epoch_start(ctx, ts, 1, False, SPEC.T_P, lg, xs, solo, g.streams[0], 20_000)
        M.check(st)
        st, stats = M.moe_p_epoch_join(runner)
        assert st == M.MOE_ERR_TIMEOUT and stats.layers_done == 0
        assert M.moe_turnstile_query(ts)[1].task == M.MOE_TS_DONE
        assert M.moe_phase_view(ctx, 0)[1].state == M.MOE_STATE_IDLE
        # the phase is still usable
        assert M.moe_p_epoch_start(ctx, ts, 1, True, SPEC.T_P, lg, xs, solo, g.streams[0], 5_000_000)[0] == \
            M.MOE_ERR_REJECTED  # stale epoch
    finally:
        M.moe_turnstile_destroy(ts)
