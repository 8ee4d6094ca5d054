"""Seeded synthetic inputs for the phase-owned MoE layer.

This module only draws inputs: router logits, hidden rows and expert
weights.  It holds none of the layer's own arithmetic (no top-k, no layout,
no FFN, no combine), and both the CPU oracle's tests and the GPU path's
tests and benchmark take their inputs from here.

Recipe (the paper's checkpoints and RL traces are internal, so these stand
in for them): every tensor block is drawn as float32 standard normals times a
scale from its own numpy PCG64 stream, seeded by SeedSequence([seed, id]):
id 0 is the router weight Wg [H, E] (std 1/sqrt(H)), ids 1..E_loc the
gate/up matrices W_gu[e] [2I, H], ids E_loc+1..2 E_loc the down matrices
W_dn[e] [H, I] (all std 1/sqrt(H)), then 2 E_loc+1 the P hidden rows [T_P, H]
and 2 E_loc+2 the D hidden rows [T_D, H] (std 1).  Separate streams let the
blocks be drawn in parallel with results independent of the thread count.  bf16 workloads round every one of them to bfloat16 (round to
nearest even) and keep the bit patterns; logits are the float32 rounding of
the float64 product of the (rounded) hidden rows with Wg, plus a per-expert
bias for skewed routing.  The logits are an input of the routing call, so
the oracle and the GPU see the very same float32 values.

FP8 workloads keep bf16 hidden rows and draw the expert weights directly in
OCP MX FP8: each block's standard normals times 16 become E4M3 codes
(PyTorch's float8_e4m3fn conversion), and each row's 32-value groups get an
E8M0 scale byte 127 + round(log2(std / 16)) + j with j drawn uniformly from
{-1, 0, 1} (so several scales occur), from the same stream.  The float32
values are the codes' values times their scales (exact).
"""

from __future__ import annotations

import concurrent.futures as cf
import dataclasses
import math
import os
from typing import Optional

import numpy as np

F32 = "f32"
BF16 = "bf16"
FP8 = "fp8"


@dataclasses.dataclass(frozen=True)
class LayerSpec:
    """Shape of one GPU's share of the layer and of its two phase batches."""

    name: str
    E: int  # expert pool size
    e0: int  # first resident expert
    E_loc: int  # resident experts
    k: int  # top-k
    H: int  # hidden size
    I: int  # FFN intermediate size
    dtype: str  # "f32", "bf16" or "fp8" (MX FP8 weights, bf16 hidden rows)
    T_P: int  # prefill batch tokens
    T_D: int  # decode batch tokens
    zipf_s: Optional[float] = None  # skewed routing exponent (None = uniform-ish)


# The named workloads.  Sizes follow the paper's model family at one GPU's
# share: a tiny fp32 check layer, a mid-size bf16 layer, a DeepSeek-V3-shaped
# expert share (32 resident of 256 routed experts, top-8, H=7168, I=2048) and
# the same share under Zipf-skewed routing.
CONFIGS = {
    0: LayerSpec("tiny-f32", E=8, e0=0, E_loc=8, k=2, H=256, I=512, dtype=F32, T_P=64, T_D=8),
    1: LayerSpec("mid-bf16", E=32, e0=0, E_loc=32, k=4, H=2048, I=1024, dtype=BF16, T_P=2048, T_D=64),
    2: LayerSpec("dsv3-share-bf16", E=256, e0=0, E_loc=32, k=8, H=7168, I=2048, dtype=BF16, T_P=8192, T_D=128),
    3: LayerSpec(
        "dsv3-share-zipf-bf16", E=256, e0=0, E_loc=32, k=8, H=7168, I=2048, dtype=BF16, T_P=16384, T_D=256, zipf_s=1.2
    ),
    # the config-2 layer under the agentic trace (agentic_trace): T_P and T_D
    # here are the token pools the trace's batches are windows of
    4: LayerSpec("dsv3-share-agentic-bf16", E=256, e0=0, E_loc=32, k=8, H=7168, I=2048, dtype=BF16, T_P=16384,
                 T_D=256),
    # the config-2 share with MX FP8 expert weights
    5: LayerSpec("dsv3-share-fp8", E=256, e0=0, E_loc=32, k=8, H=7168, I=2048, dtype=FP8, T_P=8192, T_D=128),
    # the paper's own model shape (hidden 2560, 512 routed experts, top-8)
    # at one GPU's share of EP8 (64 resident); the expert width I = 768 is a
    # reading (the paper does not state it)
    6: LayerSpec("paper-shape-fp8", E=512, e0=0, E_loc=64, k=8, H=2560, I=768, dtype=FP8, T_P=8192, T_D=256),
    7: LayerSpec("paper-shape-bf16", E=512, e0=0, E_loc=64, k=8, H=2560, I=768, dtype=BF16, T_P=8192, T_D=256),
}


def seed_of(cfg: int) -> int:
    return 1000 + cfg


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest even) and return uint16 bits.
    Inputs are finite by construction (no overflow of the 32-bit sum)."""
    u = np.ascontiguousarray(a, np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact float32 value of bfloat16 bit patterns."""
    b = np.ascontiguousarray(b, np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class LayerInputs:
    """Everything one GPU's share of the layer consumes.

    Value arrays are float32 (for bf16 workloads they hold exactly the bf16
    values); `*_bits` hold the bf16 bit patterns the GPU consumes (None for
    f32 workloads).
    """

    spec: LayerSpec
    wg: np.ndarray  # [H, E] f32
    bias: np.ndarray  # [E] f32 (zeros unless skewed)
    w_gu: np.ndarray  # [E_loc, 2I, H] f32 values
    w_dn: np.ndarray  # [E_loc, H, I] f32 values
    x: dict  # phase -> [T, H] f32 values
    logits: dict  # phase -> [T, E] f32
    w_gu_bits: Optional[np.ndarray] = None  # bf16 bits, or E4M3 codes (uint8) for fp8
    w_dn_bits: Optional[np.ndarray] = None
    x_bits: Optional[dict] = None
    w_gu_scales: Optional[np.ndarray] = None  # fp8: E8M0 bytes [E_loc, 2I, H / 32]
    w_dn_scales: Optional[np.ndarray] = None  # fp8: E8M0 bytes [E_loc, H, I / 32]


def _stream(seed: int, block: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, block])))


def _draw_mx_block(seed: int, block: int, shape, std: float):
    """One MX FP8 weight block (see the module recipe).  Returns (float32
    values, E4M3 codes uint8, E8M0 scales uint8 [..., K / 32])."""
    import torch

    rng = _stream(seed, block)
    a = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(16.0)
    codes = torch.from_numpy(a).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    base = 127 + int(round(math.log2(std / 16.0)))
    sshape = tuple(shape[:-1]) + (shape[-1] // 32,)
    scales = (base + rng.integers(-1, 2, size=sshape)).astype(np.uint8)
    vals = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float32).numpy()
    vals = (vals.reshape(sshape + (32,)) * np.exp2(scales.astype(np.float32) - 127)[..., None]).reshape(shape)
    return vals.astype(np.float32), codes, scales


def _draw_block(seed: int, block: int, shape, std: float, dtype: str):
    """One tensor block: float32 normals * std, rounded to bf16 if asked.
    Returns (float32 values, bf16 bits or None)."""
    a = _stream(seed, block).standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    if dtype == F32:
        return a, None
    bits = f32_to_bf16_bits(a)
    return bf16_bits_to_f32(bits), bits


_POOL_WORKERS = max(1, min(16, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else 4))


def logits_of(x: np.ndarray, wg: np.ndarray, bias: np.ndarray) -> np.ndarray:
    """Router logits as float32 rounding of the float64 product, plus bias."""
    if x.shape[0] == 0:
        return np.zeros((0, wg.shape[1]), np.float32)
    l = x.astype(np.float64) @ wg.astype(np.float64)
    l += bias.astype(np.float64)[None, :]
    return l.astype(np.float32)


def make_layer(spec: LayerSpec, seed: int, bias: Optional[np.ndarray] = None) -> LayerInputs:
    """Draw one layer's weights and both phase batches (see the module recipe)."""
    H, I, E, E_loc = spec.H, spec.I, spec.E, spec.E_loc
    wstd = 1.0 / math.sqrt(H)
    bf16 = spec.dtype == BF16
    fp8 = spec.dtype == FP8
    w_gu = np.empty((E_loc, 2 * I, H), np.float32)
    w_dn = np.empty((E_loc, H, I), np.float32)
    w_gu_bits = np.empty((E_loc, 2 * I, H), np.uint16) if bf16 else None
    w_dn_bits = np.empty((E_loc, H, I), np.uint16) if bf16 else None
    if fp8:
        w_gu_bits = np.empty((E_loc, 2 * I, H), np.uint8)
        w_dn_bits = np.empty((E_loc, H, I), np.uint8)
        w_gu_scales = np.empty((E_loc, 2 * I, H // 32), np.uint8)
        w_dn_scales = np.empty((E_loc, H, I // 32), np.uint8)

    def expert(job):
        kind, e = job
        if fp8:
            if kind == "gu":
                w_gu[e], w_gu_bits[e], w_gu_scales[e] = _draw_mx_block(seed, 1 + e, (2 * I, H), wstd)
            else:
                w_dn[e], w_dn_bits[e], w_dn_scales[e] = _draw_mx_block(seed, 1 + E_loc + e, (H, I), wstd)
            return
        if kind == "gu":
            v, b = _draw_block(seed, 1 + e, (2 * I, H), wstd, spec.dtype)
            w_gu[e] = v
            if bf16:
                w_gu_bits[e] = b
        else:
            v, b = _draw_block(seed, 1 + E_loc + e, (H, I), wstd, spec.dtype)
            w_dn[e] = v
            if bf16:
                w_dn_bits[e] = b

    jobs = [("gu", e) for e in range(E_loc)] + [("dn", e) for e in range(E_loc)]
    with cf.ThreadPoolExecutor(_POOL_WORKERS) as ex:
        list(ex.map(expert, jobs))
        xdt = BF16 if fp8 else spec.dtype  # FP8 layers take bf16 hidden rows
        fx = {ph: ex.submit(_draw_block, seed, 2 * E_loc + 1 + ph, ((spec.T_P, spec.T_D)[ph], H), 1.0, xdt)
              for ph in (0, 1)}
        wg = _stream(seed, 0).standard_normal(size=(H, E), dtype=np.float32) * np.float32(wstd)
        x, x_bits = {}, {}
        for ph in (0, 1):
            x[ph], x_bits[ph] = fx[ph].result()
    if bias is None:
        bias = np.zeros(E, np.float32)
    bias = np.asarray(bias, np.float32)
    logits = {ph: logits_of(x[ph], wg, bias) for ph in (0, 1)}
    return LayerInputs(
        spec=spec,
        wg=wg,
        bias=bias,
        w_gu=w_gu,
        w_dn=w_dn,
        x=x,
        logits=logits,
        w_gu_bits=w_gu_bits,
        w_dn_bits=w_dn_bits,
        x_bits=x_bits if (bf16 or fp8) else None,
        w_gu_scales=w_gu_scales if fp8 else None,
        w_dn_scales=w_dn_scales if fp8 else None,
    )


# Router biases of the skewed-routing workloads, stored as text (one float32
# per expert id).  They are calibrated offline against the CPU oracle's
# routing by tests/golden/make_zipf_bias.py, which documents the target
# shares; this module only reads them.
_ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BIAS_FILES = {3: os.path.join("tests", "golden", "zipf_bias_cfg3.txt")}


def stored_bias(cfg: int) -> np.ndarray:
    b = np.loadtxt(os.path.join(_ROOT, BIAS_FILES[cfg]), dtype=np.float64, comments="#")
    spec = CONFIGS[cfg]
    if b.shape != (spec.E,) or not np.all(np.isfinite(b)):
        raise ValueError(f"bad stored bias for config {cfg}")
    return b.astype(np.float32)


def make_config(cfg: int, seed: Optional[int] = None, bias: Optional[np.ndarray] = None) -> LayerInputs:
    spec = CONFIGS[cfg]
    if bias is None and cfg in BIAS_FILES:
        bias = stored_bias(cfg)
    return make_layer(spec, seed_of(cfg) if seed is None else seed, bias=bias)


@dataclasses.dataclass(frozen=True)
class TraceStep:
    """One step of the agentic rollout trace: a D batch of t_d tokens taken
    from the D pool at d_off, and (when t_p > 0) a continuation-prefill P
    batch of t_p tokens taken from the P pool at p_off."""

    t_d: int
    d_off: int
    t_p: int
    p_off: int


def agentic_trace(steps: int = 200, seed: int = 1004, pool_p: int = 16384, pool_d: int = 256):
    """The seeded agentic multi-turn rollout trace: each step runs a D batch
    of U{32..256} tokens and, with probability 0.5, a P batch whose size is
    log-uniform on [512, 16384] (rounded).  Batches are windows of fixed
    token pools at seeded offsets, so replaying the trace draws nothing."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out = []
    for _ in range(steps):
        t_d = int(rng.integers(32, 257))
        t_p = int(round(math.exp(rng.uniform(math.log(512), math.log(16384))))) if rng.random() < 0.5 else 0
        t_p = min(t_p, pool_p)
        d_off = int(rng.integers(0, pool_d - t_d + 1))
        p_off = int(rng.integers(0, pool_p - t_p + 1)) if t_p else 0
        out.append(TraceStep(t_d, d_off, t_p, p_off))
    return out


def tie_logits(rng: np.random.Generator, T: int, E: int, levels: int = 4) -> np.ndarray:
    """Logits drawn from a few discrete levels (with both signed zeros), so
    that many experts of a token tie; used to exercise tie-breaking."""
    vals = np.array([-1.5, -0.0, 0.0, 0.75, 2.0, 2.0, 3.25][: max(levels, 3)], np.float32)
    return rng.choice(vals, size=(T, E)).astype(np.float32)
