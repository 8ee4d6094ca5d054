"""GPU parity at the full sizes of the named workloads, through the C ABI.

Workloads: the DeepSeek-V3-shaped expert share (32 of 256 experts resident,
top-8, H = 7168, I = 2048: config 2), the same share under capped-Zipf
routing with twice the tokens (config 3), the paper's own model shape at one
GPU's share of EP8 (hidden 2560, 512 experts, 64 resident, top-8; Section
7.1) in bf16 (config 7) and MX FP8 (config 6), and config 2's share in MX
FP8 (config 5).  P and D are enqueued together on their two streams, with
D-first admission on (the bench's 500 us bound), so P's grouped-GEMM tiles
take their window checks while D runs beside them.

Checked against the oracle:
* routing, layout and x_perm exactly, for every token and row;
* h and y element by element on a set of rows that covers every m-tile of
  every expert (tests.gpu_util.covering_rows: each segment's first and last
  row and two rows around every 32nd row), with every column of each row;
* the layer output on a seeded sample of tokens: uniformly drawn ones (their
  output RMS stands for the phase's) and ones that own covering rows;
* exact zeros for every token with no resident slot.
A row's h and y and a token's output depend on no other row or token, so the
oracle runs on the sampled rows and tokens alone.
"""

import numpy as np
import pytest

import oracle
from oracle import mx as OX
from synth import make_config
from tests.test_gpu_fp8 import ACC, h_bound
from tests.gpu_util import (GpuLayer, assert_route_layout_exact, check_out_sampled, check_rows_h_y, covering_rows,
                            rms, sample_tokens, sub_offsets)

pytestmark = pytest.mark.gpu

D_PRIORITY_US = 500


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def oracle_layout(inp, ph):
    spec = inp.spec
    idx, w = oracle.route(inp.logits[ph], spec.k)
    le = oracle.local_map(idx, spec.e0, spec.E_loc)
    counts, offsets, ros, tor = oracle.layout(le, spec.E_loc)
    return dict(topk_idx=idx, topk_w=w, counts=counts, offsets=offsets, row_of_slot=ros, token_of_row=tor)


def run_concurrent(inp):
    g = GpuLayer(inp, d_priority_us=D_PRIORITY_US)
    g.run(0)
    g.run(1)
    return g


def check_bf16_phase(g, inp, ph, what):
    spec = inp.spec
    res = g.fetch(ph)
    ref = oracle_layout(inp, ph)
    assert_route_layout_exact(res, ref, what)
    tor, ros = ref["token_of_row"], ref["row_of_slot"]
    assert np.array_equal(res["x_perm_raw"], inp.x_bits[ph][tor]), f"{what} x_perm"
    none = np.all(ros < 0, axis=1)
    assert np.all(res["out"][none] == 0), f"{what} tokens with no resident slot"
    rows = covering_rows(ref["offsets"])
    print(f"[full] {what}: {res['R']} rows, checking h and y on {rows.size} covering rows", flush=True)
    check_rows_h_y(res, inp, ph, rows, ref["offsets"], tor, what)
    T = inp.logits[ph].shape[0]
    uni, own = sample_tokens(T, tor[rows], 64, 128, seed=500 + ph)
    r = check_out_sampled(res, inp, ph, uni, own, 2e-2, f"{what} out")
    print(f"[full] {what}: out max|err| = {r:.2e} x RMS on {np.union1d(uni, own).size} tokens", flush=True)


@pytest.mark.parametrize("cfg", [2, 3, 7])
def test_bf16_full_size(cfg):
    inp = make_config(cfg)
    print(f"[full] config {cfg}: {inp.spec}", flush=True)
    g = run_concurrent(inp)
    try:
        for ph in (0, 1):
            check_bf16_phase(g, inp, ph, f"cfg{cfg} phase {ph}")
    finally:
        g.close()


# ---- MX FP8 (configs 5 and 6), checked as tests/test_gpu_fp8.py does, on the
# covering rows: x codes and scales exactly; h within half an E4M3 step at
# the GPU's block scale (or the clip) plus the accumulation bound; y on the
# GPU's own h within the accumulation bound; the combine on the GPU's own y
# within float32 rounding of its k terms; the output's RMS difference from
# the FP8 oracle on the sampled tokens within 2e-2 of the output RMS.

_E4M3 = OX.e4m3_decode(np.arange(256, dtype=np.uint8))  # the oracle's decode of every code


def dequant(codes, scales):
    """The oracle's MX dequantization (oracle.mx.mx_dequantize), evaluated
    through a table of its E4M3 decode of all 256 codes: the same values,
    fast enough for full-size weight blocks."""
    c = np.asarray(codes, np.uint8)
    K = c.shape[-1]
    v = _E4M3[c].reshape(c.shape[:-1] + (K // 32, 32))
    return (v * np.exp2(np.asarray(scales, np.float64) - 127.0)[..., None]).reshape(c.shape)


class LazyMx:
    """[E_loc, N, K] dequantized MX weights, one expert at a time (the last
    expert is kept), so the oracle's per-expert loops never hold the whole
    float64 block."""

    def __init__(self, codes, scales):
        self.codes, self.scales = codes, scales
        self.shape = codes.shape
        self._e, self._v = -1, None

    def expert(self, e):
        if e != self._e:
            self._e, self._v = e, dequant(self.codes[e], self.scales[e])
        return self._v

    def __getitem__(self, key):
        if isinstance(key, tuple):
            return self.expert(int(key[0]))[key[1:]]
        return self.expert(int(key))


def check_fp8_phase(g, inp, ph, what):
    spec = inp.spec
    I = spec.I
    res = g.fetch(ph)
    ref = oracle_layout(inp, ph)
    assert_route_layout_exact(res, ref, what)
    tor, ros, off = ref["token_of_row"], ref["row_of_slot"], ref["offsets"]
    none = np.all(ros < 0, axis=1)
    assert np.all(res["out"][none] == 0), f"{what} tokens with no resident slot"
    rows = covering_rows(off)
    print(f"[full] {what}: {res['R']} rows, checking h and y on {rows.size} covering rows", flush=True)
    xc, xs = OX.mx_quantize(np.asarray(inp.x[ph][tor[rows]], np.float64))
    assert np.array_equal(res["x_scales"][rows], xs), f"{what} x scales"
    assert np.array_equal(res["x_codes"][rows], xc), f"{what} x codes"
    so = sub_offsets(rows, off)
    xq = dequant(res["x_codes"][rows], res["x_scales"][rows])
    hq = dequant(res["h_codes"][rows], res["h_scales"][rows])
    wgu = LazyMx(inp.w_gu_bits, inp.w_gu_scales)
    wdn = LazyMx(inp.w_dn_bits, inp.w_dn_scales)
    worst_h = worst_y = 0.0
    for e in range(spec.E_loc):
        a, b = int(so[e]), int(so[e + 1])
        if a == b:
            continue
        w1, w3, w2 = wgu[e, :I], wgu[e, I:], wdn[e]
        g64 = xq[a:b] @ w1.T
        u64 = xq[a:b] @ w3.T
        dg = ACC * (np.abs(xq[a:b]) @ np.abs(w1).T)
        du = ACC * (np.abs(xq[a:b]) @ np.abs(w3).T)
        sg = g64 / (1 + np.exp(-g64))
        mag = 1.1 * np.abs(u64) * dg + (np.abs(sg) + 1.1 * dg) * du
        h64 = sg * u64
        bound = h_bound(h64, res["h_scales"][rows[a:b]], mag)
        err = np.abs(hq[a:b] - h64)
        worst_h = max(worst_h, float((err / bound).max()))
        assert (err <= bound).all(), f"{what} h expert {e}: worst {float((err / bound).max()):.3g} x bound"
        y64 = hq[a:b] @ w2.T
        yb = ACC * (np.abs(hq[a:b]) @ np.abs(w2).T) + 1e-30
        ye = np.abs(res["y"][rows[a:b]] - y64)
        worst_y = max(worst_y, float((ye / yb).max()))
        assert (ye <= yb).all(), f"{what} y expert {e}: worst {float((ye / yb).max()):.3g} x bound"
    T = inp.logits[ph].shape[0]
    uni, own = sample_tokens(T, tor[rows], 64, 128, seed=600 + ph)
    toks = np.union1d(uni, own)
    # the combine on the GPU's own y, for the sampled tokens
    w_t, ros_t = ref["topk_w"][toks], ros[toks]
    comb = oracle.combine(res["y"], w_t, ros_t, toks.size, spec.H)
    absw = np.zeros_like(comb)
    for j in range(spec.k):
        r = ros_t[:, j]
        ok = r >= 0
        absw[ok] += np.abs(w_t[ok, j])[:, None] * np.abs(res["y"][r[ok]].astype(np.float64))
    assert (np.abs(res["out"][toks] - comb) <= 2 * spec.k * 2.0 ** -23 * absw + 1e-30).all(), f"{what} combine"
    # end to end against the FP8 oracle on the sampled sub-batch
    sub_out = fp8_oracle_out(inp, ph, toks, wgu, wdn)
    scale = rms(sub_out[np.searchsorted(toks, uni)])
    d_rms = rms(res["out"][toks] - sub_out) / max(scale, 1e-30)
    print(f"[full] {what}: h within {worst_h:.2f} and y within {worst_y:.2f} of their bounds; out RMS difference "
          f"{d_rms:.2e} of the output RMS on {toks.size} tokens", flush=True)
    assert d_rms <= 2e-2, f"{what} out: RMS difference {d_rms:.3e}"


def fp8_oracle_out(inp, ph, toks, wgu, wdn):
    """The FP8 oracle layer (oracle.mx.layer_mx's steps) on a sub-batch of
    tokens, with the weights dequantized one expert at a time."""
    spec = inp.spec
    lg = inp.logits[ph][toks]
    x = np.asarray(inp.x[ph][toks], np.float64)
    idx, w = oracle.route(lg, spec.k)
    le = oracle.local_map(idx, spec.e0, spec.E_loc)
    counts, offsets, ros, tor = oracle.layout(le, spec.E_loc)
    xp_codes, xp_scales = OX.mx_quantize(oracle.permute(x, tor))
    xq = OX.mx_dequantize(xp_codes, xp_scales)
    h64, h_codes, h_scales, y = OX.expert_ffn_mx(xq, offsets, wgu, wdn)
    return oracle.combine(y, w, ros, toks.size, spec.H)


@pytest.mark.parametrize("cfg", [5, 6])
def test_fp8_full_size(cfg):
    inp = make_config(cfg)
    print(f"[full] config {cfg}: {inp.spec}", flush=True)
    g = run_concurrent(inp)
    try:
        for ph in (0, 1):
            check_fp8_phase(g, inp, ph, f"cfg{cfg} phase {ph}")
    finally:
        g.close()
