"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Exact: topk_idx, counts, offsets, row_of_slot, token_of_row, x_perm (a bit
copy).  topk_w within 2e-6 relative.  The layer output within 2e-2 x RMS of
the oracle's output for bf16 layers and 1e-5 x RMS for float32 layers; h and
y element by element within the precision they are stored in (see
tests/gpu_util.py).  The
shapes below span several tiles, ragged tails and the degenerate cases
(k = 1, k = E, empty batch, experts with no rows, experts off this GPU)."""

import numpy as np
import pytest

import oracle
from synth import BF16, F32, LayerSpec, make_config, make_layer
from tests.gpu_util import (GpuLayer, assert_close_rms, assert_route_layout_exact, check_h_y, tol_of)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def check_phase(g, inp, ph):
    spec = inp.spec
    res = g.fetch(ph)
    ref = oracle.layer(inp.logits[ph], inp.x[ph], inp.w_gu, inp.w_dn, spec.k, spec.e0)
    what = f"{spec.name} phase {ph}"
    assert_route_layout_exact(res, ref, what)
    assert np.array_equal(res["x_perm"], inp.x[ph][ref["token_of_row"]]), f"{what} x_perm"
    check_h_y(res, ref, inp.w_dn, ref["offsets"], spec, what)
    assert_close_rms(res["out"], ref["out"], tol_of(spec), f"{what} out")
    # tokens without a resident slot are exact zeros
    none = np.all(ref["row_of_slot"] < 0, axis=1)
    assert np.all(res["out"][none] == 0)
    return res


SPECS = {
    "cfg0-tiny-f32": lambda: make_config(0),
    "cfg1-mid-bf16": lambda: make_config(1),
    # E not a multiple of 64, e0 > 0, I and H not multiples of the n-tiles,
    # a ragged token count, large-batch tiles for P and small-batch for D
    "ragged-bf16": lambda: make_layer(LayerSpec("ragged-bf16", E=40, e0=5, E_loc=16, k=3, H=192, I=320, dtype=BF16,
                                                T_P=1001, T_D=7), seed=11),
    # small batches only (both phases on the weight-streaming tiles)
    "skinny-bf16": lambda: make_layer(LayerSpec("skinny-bf16", E=64, e0=32, E_loc=32, k=2, H=256, I=128, dtype=BF16,
                                                T_P=50, T_D=3), seed=12),
    "k1-bf16": lambda: make_layer(LayerSpec("k1-bf16", E=16, e0=0, E_loc=16, k=1, H=128, I=128, dtype=BF16, T_P=900,
                                            T_D=2), seed=13),
    # very large batch (>= 512 rows per expert on average): 256-row tiles for
    # P, with ragged expert tails, a partial gate/up n-tile and dropped slots
    "wide-bf16": lambda: make_layer(LayerSpec("wide-bf16", E=8, e0=2, E_loc=4, k=2, H=256, I=192, dtype=BF16,
                                              T_P=2500, T_D=5), seed=15),
    # the 256-row tiles over one and two 64-deep K slices: the shortest
    # pipelines of GEMM1's ring, whose activation slices run one ahead
    "wide-k64-bf16": lambda: make_layer(LayerSpec("wide-k64-bf16", E=4, e0=0, E_loc=4, k=1, H=64, I=128, dtype=BF16,
                                                  T_P=2100, T_D=3), seed=16),
    "wide-k128-bf16": lambda: make_layer(LayerSpec("wide-k128-bf16", E=4, e0=0, E_loc=4, k=1, H=128, I=192,
                                                   dtype=BF16, T_P=2100, T_D=3), seed=17),
    # GEMM1's 256-row tiles in super-rows: 32 n-tiles (the last one partial)
    # give super-rows of 8 m-tiles, over experts of nine or ten m-tiles
    "wide-super-bf16": lambda: make_layer(LayerSpec("wide-super-bf16", E=2, e0=0, E_loc=2, k=1, H=64, I=4032,
                                                    dtype=BF16, T_P=4700, T_D=3), seed=18),
    # k = E: every expert takes every token
    "k-eq-E-bf16": lambda: make_layer(LayerSpec("kE-bf16", E=4, e0=0, E_loc=4, k=4, H=64, I=64, dtype=BF16, T_P=129,
                                                T_D=1), seed=14),
    # a pool above 256 experts (8 logits per lane), 64 resident, top-8
    "wide-pool-bf16": lambda: make_layer(LayerSpec("wide-bf16", E=300, e0=100, E_loc=64, k=8, H=128, I=192,
                                                   dtype=BF16, T_P=700, T_D=5), seed=15),
    # skewed routing on the large-batch tiles: experts of 7 to 841 rows, so
    # one to six m-tiles each, with rows that do not divide evenly among them
    "split-bf16": lambda: make_layer(LayerSpec("split-bf16", E=16, e0=0, E_loc=16, k=2, H=256, I=320, dtype=BF16,
                                               T_P=2000, T_D=6), seed=19,
                                     bias=np.linspace(1.2, -1.2, 16).astype(np.float32)),
    # the limits: 1024 experts, 256 resident, top-16; P's layout at the
    # 8192-cell bound (32 chunks x 256 experts), D's at the one-chunk bound
    # (2048 slots)
    "limits-bf16": lambda: make_layer(LayerSpec("limits-bf16", E=1024, e0=512, E_loc=256, k=16, H=128, I=128,
                                                dtype=BF16, T_P=4096, T_D=128), seed=24),
    # the longest rows: H = 16384 (GEMM1's K), then I = 16384 (GEMM2's K).
    # All experts resident and I = 128 for the first: rounding h to bf16
    # (GEMM2's operand; the oracle keeps it in float64) alone moves single
    # outputs by up to 2.8 % of the output RMS with I = 64 and three of four
    # experts elsewhere (zero rows dilute the RMS), by 1.3 % here
    "max-h-bf16": lambda: make_layer(LayerSpec("max-h-bf16", E=4, e0=0, E_loc=4, k=1, H=16384, I=128, dtype=BF16,
                                               T_P=300, T_D=5), seed=25),
    "max-i-bf16": lambda: make_layer(LayerSpec("max-i-bf16", E=4, e0=1, E_loc=1, k=1, H=64, I=16384, dtype=BF16,
                                               T_P=300, T_D=5), seed=26),
    "ragged-f32": lambda: make_layer(LayerSpec("ragged-f32", E=12, e0=3, E_loc=6, k=2, H=192, I=128, dtype=F32,
                                               T_P=77, T_D=0), seed=16),
}


@pytest.mark.parametrize("name", list(SPECS))
def test_layer_parity(name):
    inp = SPECS[name]()
    print(f"[parity] {name}: {inp.spec}", flush=True)
    g = GpuLayer(inp)
    try:
        for ph in (0, 1):
            g.run(ph)
        for ph in (0, 1):
            check_phase(g, inp, ph)
    finally:
        g.close()


def _snapshot(g, ph):
    res = g.fetch(ph)
    return {k: v.copy() for k, v in res.items() if isinstance(v, np.ndarray)}


@pytest.mark.parametrize("d_priority_us", [0, 200])
def test_concurrent_phases_bit_identical_to_solo(d_priority_us):
    """P and D enqueued on two streams at once give the same bits as each
    phase run alone: the phases share only read-only weights, and D-first
    admission only delays P's tiles."""
    import torch

    inp = make_config(1)
    g = GpuLayer(inp, d_priority_us=d_priority_us)
    try:
        g.run(0)
        p_solo = _snapshot(g, 0)
        g.run(1)
        d_solo = _snapshot(g, 1)
        for rep in range(3):
            g.run(0)
            g.run(1)
            torch.cuda.synchronize()
            p, d = _snapshot(g, 0), _snapshot(g, 1)
            for key in p_solo:
                assert np.array_equal(p[key], p_solo[key]), (rep, "P", key)
                assert np.array_equal(d[key], d_solo[key]), (rep, "D", key)
        check_phase(g, inp, 0)
        check_phase(g, inp, 1)
    finally:
        g.close()


@pytest.mark.parametrize("name", ["wide-bf16", "wide-k64-bf16", "wide-super-bf16"])
def test_wide_gemm2_share_form(name):
    """P's 256-row GEMM2 takes its share form (32-deep slices, room for D's
    decode tiles on each CU) once D-first admission is on and the context has
    run a D layer.  Both forms add the K products in the same order, so P
    gives the same bits before D's first layer (64-deep form) and after it
    (share form), and both pass the oracle checks."""
    inp = SPECS[name]()
    g = GpuLayer(inp, d_priority_us=500)
    try:
        g.run(0)  # no D layer yet: the 64-deep form
        first = _snapshot(g, 0)
        check_phase(g, inp, 0)
        g.run(1)
        g.run(0)  # the share form
        second = _snapshot(g, 0)
        for key in first:
            assert np.array_equal(first[key], second[key]), key
        check_phase(g, inp, 0)
        check_phase(g, inp, 1)
    finally:
        g.close()


def _poison_y(g, ph):
    """Fill the phase's y with NaN bits, so a tile no kernel wrote shows."""
    import ctypes

    import torch

    from tests.gpu_util import hip

    torch.cuda.synchronize()
    st, v = g.M.moe_phase_view(g.ctx, ph)
    g.M.check(st)
    h = hip()
    h.hipMemset.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t]
    h.hipMemset.restype = ctypes.c_int
    assert h.hipMemset(v.y, 0xFF, v.rows_capacity * g.spec.H * 4) == 0
    torch.cuda.synchronize()


@pytest.mark.parametrize("name", ["wide-bf16", "wide-k64-bf16"])
def test_wide_gemm2_handover(name):
    """With D-first admission on and a D layer run, P's 256-row GEMM2 is a
    hand-over pair: a launch of the full tiles does every tile that starts
    while D has no layer in flight, and a launch of the share form does the
    rest.  With D idle the first launch does them all; with D's window held
    open (D's route enqueued, the rest of its layer not) the second does.
    y is poisoned before each P layer, so a tile that neither launch did
    would show; every run gives the bits of the full form alone."""
    inp = SPECS[name]()
    g = GpuLayer(inp, d_priority_us=500)
    M = g.M
    try:
        g.run(0)  # no D layer yet: the full form alone
        ref = _snapshot(g, 0)
        g.run(1)
        for held in (False, True, False):
            if held:
                M.check(M.moe_route(g.ctx, 1, g.logits[1], g.T[1], g.streams[1]))
            _poison_y(g, 0)
            g.run(0)
            got = _snapshot(g, 0)
            for key in ref:
                assert np.array_equal(ref[key], got[key]), (held, key)
            if held:
                M.check(M.moe_phase_reset(g.ctx, 1))
                g.run(1)  # a whole D layer closes the window again
        check_phase(g, inp, 0)
        check_phase(g, inp, 1)
    finally:
        g.close()


def test_abandoned_d_window_is_not_honoured():
    """A D layer abandoned after its route leaves its window open on the
    device; after moe_phase_reset the P phase no longer waits for it (the
    reset moves D to a new window generation).  P still gives the oracle's
    result, and well inside the time a wait on every tile would take."""
    import time

    import torch

    inp = make_config(1)
    g = GpuLayer(inp, d_priority_us=1000)
    try:
        M = g.M
        g.run(0)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        g.run(0)
        torch.cuda.synchronize()
        base = time.perf_counter() - t0
        s = g.streams[1]
        M.check(M.moe_route(g.ctx, 1, g.logits[1], g.T[1], s))
        torch.cuda.synchronize()
        M.check(M.moe_phase_reset(g.ctx, 1))
        t0 = time.perf_counter()
        g.run(0)
        torch.cuda.synchronize()
        after = time.perf_counter() - t0
        # a wait on every tile would add at least 1 ms per round of tiles
        assert after < base + 2e-3, (base, after)
        check_phase(g, inp, 0)
    finally:
        g.close()


def test_open_d_window_costs_p_at_most_one_budget_per_tile():
    """A D window left open (D's route enqueued, the rest of its layer not)
    holds each P GEMM tile back for at most about d_priority_us in all: the
    tile-start and in-tile waits share one budget.  At the mid layer each
    GEMM runs two rounds of tiles, so P's layer may grow by about
    4 x 100 us; a budget per wait (nine waits per GEMM1 tile, five per
    GEMM2 tile) would allow about 2.8 ms.  P still gives the oracle's
    result."""
    import time

    import torch

    inp = make_config(1)
    g = GpuLayer(inp, d_priority_us=100)
    try:
        M = g.M
        g.run(0)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        g.run(0)
        torch.cuda.synchronize()
        base = time.perf_counter() - t0
        s = g.streams[1]
        M.check(M.moe_route(g.ctx, 1, g.logits[1], g.T[1], s))
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        g.run(0)
        torch.cuda.synchronize()
        held = time.perf_counter() - t0
        print(f"[window] P layer {base * 1e6:.0f} us, with D's window open {held * 1e6:.0f} us", flush=True)
        assert held < base + 1.2e-3, (base, held)
        check_phase(g, inp, 0)
        M.check(M.moe_phase_reset(g.ctx, 1))
    finally:
        g.close()


@pytest.mark.parametrize("name", ["cfg1-mid-bf16", "ragged-bf16"])
def test_decode_tiles_staged_and_direct_bit_identical(name):
    """D's decode tiles load their operands through an LDS stage, except
    while the other phase's latest FFN ran 160-row prefill tiles (they leave
    too little LDS), when they load straight into registers.  D alone takes
    the first, D after such a P the second: both must give the same bits
    (same MFMAs in the same order) and match the oracle."""
    inp = SPECS[name]()
    g = GpuLayer(inp)
    try:
        g.run(1)  # P has not run: staged decode tiles
        staged = _snapshot(g, 1)
        check_phase(g, inp, 1)
        g.run(0)  # P on 160-row tiles
        g.run(1)  # direct decode tiles
        direct = _snapshot(g, 1)
        for key in staged:
            assert np.array_equal(staged[key], direct[key]), key
        check_phase(g, inp, 1)
    finally:
        g.close()


def test_phase_isolation():
    """Running P never writes D's buffers (and the reverse): both phases own
    disjoint allocations."""
    inp = make_layer(LayerSpec("iso", E=16, e0=0, E_loc=16, k=2, H=128, I=128, dtype=BF16, T_P=400, T_D=9), seed=21)
    g = GpuLayer(inp)
    try:
        M = g.M
        g.run(1)
        d0 = _snapshot(g, 1)
        g.run(0)
        d1 = _snapshot(g, 1)
        for key in d0:
            assert np.array_equal(d0[key], d1[key]), key
        _, vp = M.moe_phase_view(g.ctx, 0)
        _, vd = M.moe_phase_view(g.ctx, 1)
        p_ptrs = [vp.topk_idx, vp.topk_w, vp.counts, vp.offsets, vp.row_of_slot, vp.token_of_row, vp.x_perm, vp.h, vp.y]
        d_ptrs = [vd.topk_idx, vd.topk_w, vd.counts, vd.offsets, vd.row_of_slot, vd.token_of_row, vd.x_perm, vd.h, vd.y]
        p_lo, p_hi = min(p_ptrs), max(p_ptrs)
        d_lo, d_hi = min(d_ptrs), max(d_ptrs)
        assert p_hi < d_lo or d_hi < p_lo
        # D's addresses are fixed for the context's lifetime
        g.run(1)
        _, vd2 = M.moe_phase_view(g.ctx, 1)
        assert (vd2.x_perm, vd2.h, vd2.y) == (vd.x_perm, vd.h, vd.y)
    finally:
        g.close()


def test_repeat_is_deterministic():
    inp = make_layer(LayerSpec("det", E=32, e0=0, E_loc=32, k=4, H=256, I=256, dtype=BF16, T_P=777, T_D=13), seed=22)
    g = GpuLayer(inp)
    try:
        g.run(0)
        a = _snapshot(g, 0)
        g.run(0)
        b = _snapshot(g, 0)
        for key in a:
            assert np.array_equal(a[key], b[key]), key
    finally:
        g.close()


def test_state_machine_and_errors():
    import torch

    inp = make_layer(LayerSpec("sm", E=8, e0=0, E_loc=8, k=2, H=64, I=64, dtype=BF16, T_P=32, T_D=4), seed=23)
    g = GpuLayer(inp)
    M = g.M
    try:
        ctx, s = g.ctx, g.streams[0]
        x, out, lg = g.x[0], g.out[0], g.logits[0]
        assert M.moe_dispatch(ctx, 0, x, s) == M.MOE_ERR_STATE
        assert M.moe_expert_ffn(ctx, 0, s) == M.MOE_ERR_STATE
        assert M.moe_combine(ctx, 0, out, s) == M.MOE_ERR_STATE
        assert M.moe_route(ctx, 2, lg, 32, s) == M.MOE_ERR_INVALID_PHASE
        assert M.moe_route(ctx, -1, lg, 32, s) == M.MOE_ERR_INVALID_PHASE
        assert M.moe_route(ctx, 0, lg, 33, s) == M.MOE_ERR_CAPACITY
        assert M.moe_route(ctx, 1, g.logits[1], 5, s) == M.MOE_ERR_CAPACITY
        assert M.moe_route(ctx, 0, lg, -1, s) == M.MOE_ERR_INVALID_ARG
        assert M.moe_route(ctx, 0, 0, 32, s) == M.MOE_ERR_INVALID_ARG
        assert M.moe_route(ctx, 0, lg, 32, 0) == M.MOE_ERR_INVALID_ARG  # no null stream
        assert M.moe_route(ctx, 0, lg, 32, s) == M.MOE_OK
        assert M.moe_route(ctx, 0, lg, 32, s) == M.MOE_ERR_STATE  # one pending op per phase
        assert M.moe_phase_view(ctx, 0)[1].state == M.MOE_STATE_ROUTED
        assert M.moe_phase_view(ctx, 1)[1].state == M.MOE_STATE_IDLE  # D untouched
        assert M.moe_dispatch(ctx, 0, 0, s) == M.MOE_ERR_INVALID_ARG
        assert M.moe_dispatch(ctx, 0, x, s) == M.MOE_OK
        # cancellation: reset once the phase's work completed
        torch.cuda.synchronize()
        assert M.moe_phase_reset(ctx, 0) == M.MOE_OK
        assert M.moe_phase_view(ctx, 0)[1].state == M.MOE_STATE_IDLE
        # an empty batch is a legal no-work call and advances the phase
        M.check(M.moe_route(ctx, 1, 0, 0, s))
        M.check(M.moe_dispatch(ctx, 1, 0, s))
        M.check(M.moe_expert_ffn(ctx, 1, s))
        M.check(M.moe_combine(ctx, 1, 0, s))
        torch.cuda.synchronize()
        _, v = M.moe_phase_view(ctx, 1)
        assert v.state == M.MOE_STATE_IDLE and v.tokens == 0
        # a phase driven across two streams stays ordered
        s2 = g.streams[1]
        M.check(M.moe_route(ctx, 0, lg, 32, s))
        M.check(M.moe_dispatch(ctx, 0, x, s2))
        M.check(M.moe_expert_ffn(ctx, 0, s))
        M.check(M.moe_combine(ctx, 0, out, s2))
        check_phase(g, inp, 0)
        # timing records
        M.check(M.moe_timing_enable(ctx, 8))
        g.run(0)
        torch.cuda.synchronize()
        st, ms, n = M.moe_timing_read(ctx, 0, M.MOE_KERNEL_GEMM1)
        assert st == 0 and n == 1 and ms > 0
        st, ms, n = M.moe_timing_read(ctx, 0, M.MOE_KERNEL_GEMM1)
        assert st == 0 and n == 0
        M.check(M.moe_timing_enable(ctx, 0))
    finally:
        g.close()


def test_clock_probe_reads_a_plausible_clock():
    """The engine clock probe spins for the requested reference time and
    reports shader-clock ticks that give a clock between 0.2 and 4 GHz."""
    import torch

    from paper_2609_00993_amd import moepd as M

    buf = torch.zeros(2, dtype=torch.int64, device="cuda")
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    M.check(M.moe_clock_probe(s, 300, buf.data_ptr()), "moe_clock_probe")
    torch.cuda.synchronize()
    ticks, ref = buf.tolist()
    assert ref >= 300 * 100, ref
    mhz = ticks * 100.0 / ref
    print(f"[clock] {mhz:.0f} MHz", flush=True)
    assert 200 <= mhz <= 4000, mhz
