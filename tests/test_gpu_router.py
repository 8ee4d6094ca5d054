"""GPU: gating from hidden states (moe_route_from_hidden), through the C ABI.

Checks, per phase:
  * logits: the GPU's float32 logits against the oracle's float64
    x Wr^T (+ bias) on the same input values, element by element, within the
    rounding bound of a float32 sum of H exact products plus the split
    partial sums and the bias add: gamma_n sum_h |x_h w_h| (+ |bias|) with
    n = H + splits + 1 and gamma_n = n u / (1 - n u), u = 2^-24;
  * top-k: topk_idx exactly as the oracle's top-k of the GPU's own logits
    (both decide on the same float32 values), topk_w within 2e-6 relative;
  * flips against the oracle's float64 logits are counted, and each must be
    a near tie: the selection boundary's two logits within twice the bound;
  * the layer that follows (dispatch, FFN, combine) against the oracle layer
    on the GPU's logits, to the usual output tolerance.
Router weights are the generator's gate matrix, transposed to [E, H] and,
for bf16 contexts, rounded to bf16 (the oracle takes the rounded values)."""

import numpy as np
import pytest

import oracle
from oracle import mx as OX
from synth import BF16, F32, FP8, LayerSpec, f32_to_bf16_bits, bf16_bits_to_f32, make_config, make_layer
from tests.gpu_util import GpuLayer, W_RTOL, assert_close_rms, read_dev, rms, to_dev, tol_of

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


SPECS = {
    "cfg0-tiny-f32": lambda: make_config(0),
    "cfg1-mid-bf16": lambda: make_config(1),
    # E not a multiple of 64 (nor of the 128-expert n-tile), ragged T
    "ragged-bf16": lambda: make_layer(LayerSpec("ragged-bf16", E=40, e0=5, E_loc=16, k=3, H=192, I=320, dtype=BF16,
                                                T_P=1001, T_D=7), seed=11),
    # E not a multiple of 4, a pool above 256 experts
    "odd-pool-bf16": lambda: make_layer(LayerSpec("odd-pool-bf16", E=301, e0=100, E_loc=64, k=8, H=256, I=192,
                                                  dtype=BF16, T_P=300, T_D=5), seed=17),
    "ragged-f32": lambda: make_layer(LayerSpec("ragged-f32", E=12, e0=3, E_loc=6, k=2, H=192, I=128, dtype=F32,
                                               T_P=77, T_D=0), seed=16),
    # FP8 contexts gate on bf16 hidden states with a bf16 gate matrix
    "fp8": lambda: make_layer(LayerSpec("fp8", E=40, e0=5, E_loc=16, k=3, H=256, I=384, dtype=FP8, T_P=700,
                                        T_D=7), seed=18),
}

U = 2.0 ** -24


def router_inputs(inp, with_bias):
    """Gate matrix as [E, H] in the context dtype: device array and the values
    the oracle takes."""
    wt = np.ascontiguousarray(inp.wg.T)
    if inp.spec.dtype in (BF16, FP8):
        bits = f32_to_bf16_bits(wt)
        vals = bf16_bits_to_f32(bits)
        dev = to_dev(bits)
    else:
        vals = wt
        dev = to_dev(wt)
    bias = None
    if with_bias:
        bias = np.random.default_rng(99).standard_normal(inp.spec.E).astype(np.float32) * np.float32(0.5)
    return dev, vals, bias


def check_router(g, inp, ph, w_vals, bias, splits_max=32):
    spec = inp.spec
    T, E, H, k = (spec.T_P, spec.T_D)[ph], spec.E, spec.H, spec.k
    st, v = g.M.moe_phase_view(g.ctx, ph)
    g.M.check(st)
    import torch

    torch.cuda.synchronize()
    lg = read_dev(v.logits, (T, E), np.float32)
    idx = read_dev(v.topk_idx, (T, k), np.int32)
    w = read_dev(v.topk_w, (T, k), np.float32)
    x = inp.x[ph]
    ref = oracle.router_logits(x, w_vals, bias)
    mag = np.abs(np.asarray(x, np.float64)) @ np.abs(np.asarray(w_vals, np.float64)).T
    if bias is not None:
        mag = mag + np.abs(bias.astype(np.float64))[None, :]
    n = H + splits_max + 1
    bound = n * U / (1 - n * U) * mag + 1e-30
    err = np.abs(lg.astype(np.float64) - ref)
    assert (err <= bound).all(), f"{spec.name} ph{ph}: logits off by {float((err / bound).max()):.2f} x bound"
    # top-k decided on the GPU's own logits
    ridx, rw = oracle.route(lg, k)
    assert np.array_equal(idx, ridx), f"{spec.name} ph{ph}: topk_idx"
    rel = np.abs(w.astype(np.float64) - rw) / np.maximum(np.abs(rw), 1e-30)
    assert rel.size == 0 or rel.max() <= W_RTOL
    # flips against the float64 logits are near ties
    fidx, _ = oracle.route(ref, k)
    flips = 0
    for t in np.nonzero((np.sort(fidx, axis=1) != np.sort(idx, axis=1)).any(axis=1))[0]:
        flips += 1
        srt = np.sort(ref[t])[::-1]
        gap = srt[k - 1] - srt[k]
        assert gap <= 2 * float(bound[t].max()), f"{spec.name} ph{ph} token {t}: flip with gap {gap}"
    print(f"[router] {spec.name} ph{ph}: T={T} max err/bound {float((err / bound).max()) if T else 0:.3g}, "
          f"flips {flips}", flush=True)
    return lg


@pytest.mark.parametrize("with_bias", [False, True])
@pytest.mark.parametrize("name", list(SPECS))
def test_route_from_hidden(name, with_bias):
    import torch

    inp = SPECS[name]()
    spec = inp.spec
    print(f"[router] {name} bias={with_bias}: {spec}", flush=True)
    g = GpuLayer(inp)
    try:
        M = g.M
        w_dev, w_vals, bias = router_inputs(inp, with_bias)
        b_dev = to_dev(bias) if bias is not None else None
        for ph in (0, 1):
            T = g.T[ph]
            s = g.streams[ph]
            M.check(M.moe_route_from_hidden(g.ctx, ph, g.x[ph], w_dev, b_dev, T, s), "moe_route_from_hidden")
            M.check(M.moe_dispatch(g.ctx, ph, g.x[ph], s))
            M.check(M.moe_expert_ffn(g.ctx, ph, s))
            M.check(M.moe_combine(g.ctx, ph, g.out[ph], s))
        for ph in (0, 1):
            lg = check_router(g, inp, ph, w_vals, bias)
            torch.cuda.synchronize()
            if spec.dtype == FP8:
                ref = OX.layer_mx(lg, inp.x[ph], inp.w_gu_bits, inp.w_gu_scales, inp.w_dn_bits, inp.w_dn_scales,
                                  spec.k, spec.e0)
                d = rms(g.out[ph].cpu().numpy() - ref["out"]) / max(rms(ref["out"]), 1e-30)
                assert d <= 2e-2, f"{name} ph{ph} out: RMS difference {d:.3e}"  # the FP8 layer's bar
            else:
                ref = oracle.layer(lg, inp.x[ph], inp.w_gu, inp.w_dn, spec.k, spec.e0)
                assert_close_rms(g.out[ph].cpu().numpy(), ref["out"], tol_of(spec), f"{name} ph{ph} out")
        # a second call gives the same bits (fixed split order)
        first = {ph: read_dev(M.moe_phase_view(g.ctx, ph)[1].logits, (g.T[ph], spec.E), np.float32)
                 for ph in (0, 1)}
        for ph in (0, 1):
            s = g.streams[ph]
            M.check(M.moe_route_from_hidden(g.ctx, ph, g.x[ph], w_dev, b_dev, g.T[ph], s))
            M.check(M.moe_dispatch(g.ctx, ph, g.x[ph], s))
            M.check(M.moe_expert_ffn(g.ctx, ph, s))
            M.check(M.moe_combine(g.ctx, ph, g.out[ph], s))
        torch.cuda.synchronize()
        for ph in (0, 1):
            again = read_dev(M.moe_phase_view(g.ctx, ph)[1].logits, (g.T[ph], spec.E), np.float32)
            assert np.array_equal(again.view(np.uint32), first[ph].view(np.uint32))
    finally:
        g.close()


def test_route_from_hidden_batch_sizes():
    """One context, batches from 1 token to the capacity: every K-split count
    the launcher picks, the empty batch, and the refusals."""
    import torch

    inp = make_config(1)
    spec = inp.spec
    g = GpuLayer(inp)
    try:
        M = g.M
        w_dev, w_vals, _ = router_inputs(inp, False)
        s = g.streams[0]
        for T in (1, 5, 63, 64, 65, 200, 777, spec.T_P):
            M.check(M.moe_route_from_hidden(g.ctx, 0, g.x[0], w_dev, None, T, s))
            torch.cuda.synchronize()
            st, v = M.moe_phase_view(g.ctx, 0)
            lg = read_dev(v.logits, (T, spec.E), np.float32)
            ref = oracle.router_logits(inp.x[0][:T], w_vals)
            mag = np.abs(inp.x[0][:T].astype(np.float64)) @ np.abs(w_vals.astype(np.float64)).T
            n = spec.H + 33
            assert (np.abs(lg - ref) <= n * U * 1.001 * mag).all(), T
            idx = read_dev(v.topk_idx, (T, spec.k), np.int32)
            assert np.array_equal(idx, oracle.route(lg, spec.k)[0]), T
            M.check(M.moe_phase_reset(g.ctx, 0))
        # T = 0 is a legal no-work call
        M.check(M.moe_route_from_hidden(g.ctx, 0, None, None, None, 0, s))
        torch.cuda.synchronize()
        M.check(M.moe_phase_reset(g.ctx, 0))
        # refusals: capacity, null weights, out of order
        assert M.moe_route_from_hidden(g.ctx, 0, g.x[0], w_dev, None, spec.T_P + 1, s) == M.MOE_ERR_CAPACITY
        assert M.moe_route_from_hidden(g.ctx, 0, g.x[0], None, None, 4, s) == M.MOE_ERR_INVALID_ARG
        assert M.moe_route_from_hidden(g.ctx, 0, g.x[0], w_dev, None, -1, s) == M.MOE_ERR_INVALID_ARG
        M.check(M.moe_route_from_hidden(g.ctx, 0, g.x[0], w_dev, None, 4, s))
        assert M.moe_route_from_hidden(g.ctx, 0, g.x[0], w_dev, None, 4, s) == M.MOE_ERR_STATE
        torch.cuda.synchronize()
        M.check(M.moe_phase_reset(g.ctx, 0))
    finally:
        g.close()
