"""GPU parity over seeded random layer shapes (through the C ABI).

The fixed shapes of test_gpu_layer and test_gpu_fp8 each pin one chosen
case.  These tests draw 20 more from per-seed generators, four per family:
- bf16 weight-streaming decode tiles (fewer than 32 expected rows per
  expert);
- bf16 160-row tiles;
- bf16 256-row tiles (at least 512 expected rows per expert);
- MX FP8 (either FP8 tile);
- float32.

Each draw picks:
- the pool size, the resident block and top-k;
- H and I (multiples of the dtype's granule, so partial n-tiles are
  common);
- both batch sizes (empty batches included);
- an even or skewed router bias.

Expert row counts, ragged tails, empty experts and experts off this GPU
therefore vary from seed to seed.  Odd seeds run D's layer first with
D-first admission on, so P takes the tiles it uses beside D (the 256-row
GEMM2 as a hand-over pair of the full and the share form).

The checks are the fixed shapes' own: exact routing and layout, then every
stage within the dtype's bound (h and y element by element for bf16 and
float32, the combine on the GPU's own y, the FP8 stages as in
test_gpu_fp8), with one reading for the end-to-end bar of bf16 layers.  h
is stored in bf16, as GEMM2's operand.  Rounded exactly, with every other
step in float64, that storage alone moves the output of a random shape by
up to 3.7 % of its RMS (seeds 1, 6, 12 and 17 here exceed 2 %).  A max-abs
bar against an RMS is strict where zero rows of tokens with no resident
expert dilute the RMS, or where a skewed top-1 layer has heavy-tailed
outputs.  The bar is therefore the larger of 2e-2 x RMS and 1.25 times what
exact rounding of h gives, computed here on the CPU.  The kernels' own
float32 sums and the rare h elements that round the other way on the GPU
stay well inside the margin (the test prints both figures)."""

import numpy as np
import pytest

import oracle
from oracle import moe as OM
from synth import BF16, F32, FP8, LayerSpec, make_layer
from tests.gpu_util import GpuLayer, assert_route_layout_exact, check_h_y, rms, tol_of
from tests.test_gpu_fp8 import check_phase as check_fp8

FAMILIES = ("decode", "prefill", "wide", "fp8", "f32")
SEEDS = range(20)
AVG = {"decode": (1, 31), "prefill": (32, 399), "wide": (512, 899), "fp8": (1, 299), "f32": (1, 119)}
MAX_T = 6000  # keeps the float64 oracle to seconds


@pytest.fixture(scope="module")
def need_gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def draw(seed):
    """The spec and router bias of one seed (family = seed mod 5)."""
    rng = np.random.default_rng(9100 + seed)
    fam = FAMILIES[seed % len(FAMILIES)]
    gran = 128 if fam == "fp8" else 64
    lo, hi = AVG[fam]
    while True:  # pool, top-k and batch with the family's expected rows per expert (T k / E)
        E = int(rng.choice([2, 3, 4, 6, 8] if fam == "wide" else [4, 8, 12, 40, 64, 96, 300]))
        k = int(rng.integers(1, min(E, 8) + 1))
        t_lo, t_hi = -(-lo * E // k), min(MAX_T, ((hi + 1) * E - 1) // k)
        if t_lo <= t_hi:
            break
    T_P = int(rng.integers(t_lo, t_hi + 1))
    if fam == "decode" and rng.random() < 0.3:
        T_P = 0  # an empty P batch beside a decode batch
    E_loc = int(rng.integers(1, min(E, 64) + 1))
    e0 = int(rng.integers(0, E - E_loc + 1))
    H = gran * int(rng.integers(1, 5))
    I = gran * int(rng.integers(1, 5))
    T_D = int(rng.choice([0, 1, 3, int(rng.integers(1, 40))]))
    dtype = {"fp8": FP8, "f32": F32}.get(fam, BF16)
    spec = LayerSpec(f"seed{seed}-{fam}", E=E, e0=e0, E_loc=E_loc, k=k, H=H, I=I, dtype=dtype, T_P=T_P, T_D=T_D)
    bias = None
    if rng.random() < 0.5:  # skewed: a Zipf-like ramp, popular experts first or shuffled
        bias = (-1.2 * np.log1p(np.arange(E))).astype(np.float32)
        if rng.random() < 0.3:
            rng.shuffle(bias)
    return spec, bias


def bf16_rne(a):
    """float32 -> nearest bf16 (ties to even), returned as float64."""
    b = np.asarray(a, np.float32).view(np.uint32).astype(np.uint64)
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def bf16_h_floor(inp, ref, ph):
    """max|out - oracle out| / RMS(oracle out) when only h is rounded to bf16."""
    spec, off = inp.spec, ref["offsets"]
    h = bf16_rne(ref["h"])
    y = np.zeros_like(ref["y"])
    for e in range(spec.E_loc):
        a, b = int(off[e]), int(off[e + 1])
        if a < b:
            y[a:b] = h[a:b] @ np.asarray(inp.w_dn[e], np.float64).T
    T = spec.T_P if ph == 0 else spec.T_D
    out = OM.combine(y, ref["topk_w"], ref["row_of_slot"], T, spec.H)
    return float(np.max(np.abs(out - ref["out"]))) / max(rms(ref["out"]), 1e-30)


def check_dense(g, inp, ph):
    spec = inp.spec
    res = g.fetch(ph)
    ref = oracle.layer(inp.logits[ph], inp.x[ph], inp.w_gu, inp.w_dn, spec.k, spec.e0)
    what = f"{spec.name} phase {ph}"
    assert_route_layout_exact(res, ref, what)
    assert np.array_equal(res["x_perm"], inp.x[ph][ref["token_of_row"]]), f"{what} x_perm"
    check_h_y(res, ref, inp.w_dn, ref["offsets"], spec, what)
    none = np.all(ref["row_of_slot"] < 0, axis=1)
    assert np.all(res["out"][none] == 0), f"{what}: a token with no resident slot has a nonzero row"
    if ref["out"].size == 0:
        return
    # the combine on the GPU's own y and weights: float32 products and a
    # float32 sum of k terms in slot order
    T = spec.T_P if ph == 0 else spec.T_D
    w = res["topk_w"].astype(np.float64)
    y = res["y"].astype(np.float64)
    comb = OM.combine(y, w, ref["row_of_slot"], T, spec.H)
    absw = np.zeros_like(comb)
    for j in range(spec.k):
        rows = ref["row_of_slot"][:, j]
        ok = rows >= 0
        absw[ok] += np.abs(w[ok, j])[:, None] * np.abs(y[rows[ok]])
    assert (np.abs(res["out"] - comb) <= 2 * spec.k * 2.0 ** -23 * absw + 1e-30).all(), f"{what} combine"
    err = float(np.max(np.abs(res["out"] - ref["out"]))) / max(rms(ref["out"]), 1e-30)
    bar = tol_of(spec)
    if spec.dtype == BF16 and ref["y"].shape[0] > 0:
        floor = bf16_h_floor(inp, ref, ph)
        bar = max(bar, 1.25 * floor)
        print(f"[seed] {what}: max|err| {err:.4f} x RMS; exact bf16 rounding of h alone {floor:.4f}", flush=True)
    assert err <= bar, f"{what} out: max|err| {err:.3e} x RMS > {bar:.3e}"


@pytest.mark.gpu
@pytest.mark.parametrize("seed", list(SEEDS))
def test_seeded_layer_parity(seed, need_gpu):
    spec, bias = draw(seed)
    # odd seeds: D first with D-first admission on, so P's 256-row GEMM2 runs
    # as the hand-over pair and P's 160-row tiles carry the D window word
    d_first = seed % 2 == 1
    print(f"[seed {seed}] {spec} bias={'skewed' if bias is not None else 'none'} d_first={d_first}", flush=True)
    inp = make_layer(spec, seed=500 + seed, bias=bias)
    g = GpuLayer(inp, d_priority_us=500 if d_first else 0)
    try:
        for ph in ((1, 0) if d_first else (0, 1)):
            g.run(ph)
        check = check_fp8 if spec.dtype == FP8 else check_dense
        for ph in (0, 1):
            check(g, inp, ph)
    finally:
        g.close()


def test_draws_cover_every_regime():
    """The draws hit every tile family the library picks by expected rows
    per expert (the same rule as the layout call)."""
    seen = set()
    for seed in SEEDS:
        spec, _ = draw(seed)
        avg = spec.T_P * spec.k // spec.E
        if spec.dtype == BF16:
            seen.add("wide" if avg >= 512 else "prefill" if avg >= 32 else "decode")
        elif spec.dtype == FP8:
            seen.add("fp8-prefill" if avg >= 32 else "fp8-skinny")
        else:
            seen.add("f32")
    assert seen == {"wide", "prefill", "decode", "fp8-prefill", "fp8-skinny", "f32"}, seen
