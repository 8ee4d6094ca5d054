"""GPU parity of the MX FP8 expert layer (FP8 contexts) against the oracle.

Decisions on identical values are exact: routing, layout, and the x_perm
codes and scales (both sides quantize the same bf16 values).  h is
quantized from sums the two sides form in different precisions (float32
MFMA accumulation here, float64 in the oracle), so it is checked against the
oracle's unquantized h within half an E4M3 step at the GPU's own block
scale (or the clip to 448) plus the accumulation bound.  GEMM2 is checked
on the GPU's own h: y against float64 from the same dequantized codes within
the accumulation bound, and the combine on the GPU's own y within float32
rounding of its k terms.  End to end, the RMS of the difference from the
oracle's FP8 layer stays within 2e-2 of the output's RMS: h codes near a
rounding boundary may land one E4M3 step (6.25 %) apart on the two sides,
and with I terms per output a few such flips reach 10 % of the RMS at single
elements (simulating float32-sized accumulation noise of 1e-5 sum|x w| on
the oracle flips 2 % of the codes and gives an RMS difference of 0.5 %), so
a max-abs bar would test the flips, not the kernels.  The measured distances
are printed.

Accumulation bound: the scaled MFMA adds 64 exact products per step into a
float32 accumulator; measured against float64 it stays within 2^-12 of the
step's sum of |products| (about 1.5e-4 on random E4M3 data), so the bound
used is 2^-11 * sum_k |a_k b_k| over all of K."""

import numpy as np
import pytest

from oracle import moe as OM
from oracle import mx as OX
from synth import FP8, LayerSpec, make_layer
from tests.gpu_util import GpuLayer, assert_close_rms, assert_route_layout_exact, rms

pytestmark = pytest.mark.gpu

ACC = 2.0 ** -11


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


SPECS = {
    # E not a multiple of 64, e0 > 0, ragged T, I not a multiple of the 128 n-tile
    "ragged-fp8": LayerSpec("ragged-fp8", E=40, e0=5, E_loc=16, k=3, H=256, I=384, dtype=FP8, T_P=1001, T_D=7),
    "mid-fp8": LayerSpec("mid-fp8", E=32, e0=0, E_loc=32, k=4, H=2048, I=1024, dtype=FP8, T_P=2048, T_D=64),
    "k1-fp8": LayerSpec("k1-fp8", E=16, e0=0, E_loc=16, k=1, H=128, I=128, dtype=FP8, T_P=900, T_D=2),
    "empty-d-fp8": LayerSpec("empty-d-fp8", E=12, e0=3, E_loc=6, k=2, H=384, I=256, dtype=FP8, T_P=77, T_D=0),
    # skewed routing: experts of a few to ~850 rows, several m-tiles each
    "split-fp8": LayerSpec("split-fp8", E=16, e0=0, E_loc=16, k=2, H=256, I=384, dtype=FP8, T_P=2000, T_D=6),
    # the limits: 1024 experts, 256 resident, top-16
    "limits-fp8": LayerSpec("limits-fp8", E=1024, e0=512, E_loc=256, k=16, H=128, I=128, dtype=FP8, T_P=4096,
                            T_D=128),
}
BIAS = {"split-fp8": np.linspace(1.2, -1.2, 16).astype(np.float32)}


def h_bound(h64, scales_gpu, mag):
    """Half an E4M3 step of each |h| at the GPU's block scale (or the clip),
    plus the accumulation bound carried through the SwiGLU."""
    step = np.repeat(np.exp2(scales_gpu.astype(np.float64) - 127), 32, axis=1)
    a = np.abs(h64) / step
    half = np.where(a >= 2.0 ** -6, np.exp2(np.floor(np.log2(np.maximum(a, 1e-300))) - 4), 2.0 ** -10)
    clip = np.maximum(a - 448.0, 0.0)
    return (np.maximum(half, clip) * 1.01) * step + mag


def check_phase(g, inp, ph):
    spec = inp.spec
    res = g.fetch(ph)
    ref = OX.layer_mx(inp.logits[ph], inp.x[ph], inp.w_gu_bits, inp.w_gu_scales, inp.w_dn_bits, inp.w_dn_scales,
                      spec.k, spec.e0)
    what = f"{spec.name} ph{ph}"
    assert_route_layout_exact(res, ref, what)
    # x_perm: both sides quantize the same bf16 values
    assert np.array_equal(res["x_scales"], ref["x_scales"]), f"{what} x scales"
    assert np.array_equal(res["x_codes"], ref["x_codes"]), f"{what} x codes"
    if res["R"] == 0:
        assert np.all(res["out"] == 0)
        return
    wgu = OX.mx_dequantize(inp.w_gu_bits, inp.w_gu_scales)
    wdn = OX.mx_dequantize(inp.w_dn_bits, inp.w_dn_scales)
    xq = OX.mx_dequantize(res["x_codes"], res["x_scales"])
    off = ref["offsets"]
    I = spec.I
    # h against the unquantized float64 h
    mag = np.zeros_like(ref["h64"])
    for e in range(spec.E_loc):
        a, b = int(off[e]), int(off[e + 1])
        if a == b:
            continue
        g64 = xq[a:b] @ wgu[e, :I].T
        u64 = xq[a:b] @ wgu[e, I:].T
        dg = ACC * (np.abs(xq[a:b]) @ np.abs(wgu[e, :I]).T)
        du = ACC * (np.abs(xq[a:b]) @ np.abs(wgu[e, I:]).T)
        sg = g64 / (1 + np.exp(-g64))
        mag[a:b] = 1.1 * np.abs(u64) * dg + (np.abs(sg) + 1.1 * dg) * du
    hq = OX.mx_dequantize(res["h_codes"], res["h_scales"])
    bound = h_bound(ref["h64"], res["h_scales"], mag)
    err = np.abs(hq - ref["h64"])
    assert (err <= bound).all(), f"{what} h: worst {float((err / bound).max()):.3g} x bound"
    same = float(np.mean(res["h_codes"] == ref["h_codes"]))
    # y on the GPU's own h
    for e in range(spec.E_loc):
        a, b = int(off[e]), int(off[e + 1])
        if a == b:
            continue
        y64 = hq[a:b] @ wdn[e].T
        yb = ACC * (np.abs(hq[a:b]) @ np.abs(wdn[e]).T) + 1e-30
        ye = np.abs(res["y"][a:b] - y64)
        assert (ye <= yb).all(), f"{what} y expert {e}: worst {float((ye / yb).max()):.3g} x bound"
    # combine on the GPU's own y (float32 sums of k weighted terms)
    T = spec.T_P if ph == 0 else spec.T_D
    comb = OM.combine(res["y"].astype(np.float64), ref["topk_w"], ref["row_of_slot"], T, spec.H)
    absw = np.zeros_like(comb)
    for j in range(spec.k):
        rows = ref["row_of_slot"][:, j]
        ok = rows >= 0
        absw[ok] += np.abs(ref["topk_w"][ok, j])[:, None] * np.abs(res["y"][rows[ok]].astype(np.float64))
    assert (np.abs(res["out"] - comb) <= 2 * spec.k * 2.0 ** -23 * absw + 1e-30).all(), f"{what} combine"
    d_rms = rms(res["out"] - ref["out"]) / max(rms(ref["out"]), 1e-30)
    assert d_rms <= 2e-2, f"{what} out: RMS difference {d_rms:.3e} of the output RMS"
    # informational: distance from the unquantized layer on the same weights
    full = OM.layer(inp.logits[ph], inp.x[ph], wgu, wdn, spec.k, spec.e0)["out"]
    print(f"[fp8] {what}: h codes equal to the oracle's {100 * same:.2f} %; out vs FP8 oracle: RMS diff "
          f"{d_rms:.2e}, max {float(np.max(np.abs(res['out'] - ref['out']))) / max(rms(ref['out']), 1e-30):.2e} x RMS; "
          f"vs the unquantized layer: RMS diff {rms(res['out'] - full) / max(rms(full), 1e-30):.2e}", flush=True)


@pytest.mark.parametrize("name", list(SPECS))
def test_fp8_layer_parity(name):
    spec = SPECS[name]
    print(f"[fp8] {spec}", flush=True)
    inp = make_layer(spec, seed=41, bias=BIAS.get(name))
    g = GpuLayer(inp)
    try:
        for ph in (0, 1):
            g.run(ph)
        for ph in (0, 1):
            check_phase(g, inp, ph)
    finally:
        g.close()


def test_fp8_concurrent_phases_match_solo():
    """P and D on their own streams at once give each phase's solo bits."""
    import torch

    inp = make_layer(SPECS["mid-fp8"], seed=42)
    g = GpuLayer(inp, d_priority_us=200)
    try:
        for ph in (0, 1):
            g.run(ph)
        torch.cuda.synchronize()
        solo = {ph: g.out[ph].clone() for ph in (0, 1)}
        for _ in range(3):
            g.run(0)
            g.run(1)
        torch.cuda.synchronize()
        for ph in (0, 1):
            assert torch.equal(g.out[ph], solo[ph]), ph
    finally:
        g.close()
