"""Plain CPU oracle of the FP8 expert layer: OCP MX FP8 (E4M3 elements with a
shared E8M0 scale per 32 consecutive values along K).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product path never
imports, calls or links it, and it imports nothing from the product package.

What is computed, and where it comes from
-----------------------------------------
The paper runs its rollouts on BF16 and FP8 checkpoints of the same model
(Section 7.1) and does not describe its FP8 format.  This oracle follows the
reading taken for the FP8 layer:

* weights: FP8 E4M3 codes (OCP "E4M3FN": 1 sign, 4 exponent bits with bias 7,
  3 mantissa bits; no infinities; 0x7F/0xFF are NaN; largest finite 448;
  subnormals m * 2^-9) with one E8M0 scale byte per 32 consecutive values of
  a row along K (the value of byte s is 2^(s - 127));
* activations (the permuted x rows and h): quantized to the same format per
  32 consecutive values of a row.  The block's shared exponent is
  E = floor(log2(amax)) - 8 (8 is E4M3's largest normal exponent), clamped
  to [-127, 127], or -127 when amax = 0; each value v becomes the E4M3 code
  of v / 2^E rounded to nearest, ties to even, after clamping v / 2^E to
  [-448, 448] (the block maximum lands in [256, 512), so only values above
  448 clip);
* the GEMMs multiply the dequantized values exactly (float64 here); x enters
  as bf16 values, the SwiGLU is applied to float64 g and u, and y, out are
  float64 (the GPU keeps them in float32).

Everything else (routing, layout, combine) is oracle/moe.py's.
"""

from __future__ import annotations

import numpy as np

from . import moe

__all__ = [
    "e4m3_decode",
    "e4m3_encode",
    "mx_quantize",
    "mx_dequantize",
    "expert_ffn_mx",
    "layer_mx",
]

BLOCK = 32
E4M3_MAX = 448.0
E4M3_EMAX = 8


def e4m3_decode(codes) -> np.ndarray:
    """float64 values of E4M3 codes (NaN for 0x7F and 0xFF)."""
    c = np.asarray(codes, np.uint8).astype(np.int64)
    s = (c >> 7) & 1
    e = (c >> 3) & 15
    m = c & 7
    mag = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    mag = np.where((e == 15) & (m == 7), np.nan, mag)
    return np.where(s == 1, -mag, mag)


def e4m3_encode(v) -> np.ndarray:
    """E4M3 code of each value: round to nearest, ties to even; values beyond
    448 in magnitude saturate to +-448; the sign of a zero result is kept."""
    v = np.asarray(v, np.float64)
    sign = np.signbit(v).astype(np.int64) << 7
    a = np.minimum(np.abs(v), E4M3_MAX)
    code = np.zeros(a.shape, np.int64)
    # subnormal range (and zero): multiples of 2^-9 below 2^-6
    sub = a < 2.0 ** -6
    q = np.round(a[sub] * 2.0 ** 9)  # numpy rounds half to even
    code[sub] = q.astype(np.int64)  # q = 8 is the smallest normal, code 0x08
    # normal range: 1.m * 2^e, e in [-6, 8]
    nrm = ~sub
    mant, exp = np.frexp(a[nrm])  # a = mant * 2^exp, mant in [0.5, 1)
    e = exp - 1
    m = np.round((mant * 2.0 - 1.0) * 8.0).astype(np.int64)
    carry = m == 8
    e = np.where(carry, e + 1, e)
    m = np.where(carry, 0, m)
    code[nrm] = ((e + 7) << 3) | m
    return (code | sign).astype(np.uint8)


def _block_exponent(amax: np.ndarray) -> np.ndarray:
    """Shared exponent of each block from its largest magnitude (floor(log2)
    taken from frexp, which is exact)."""
    mant, exp = np.frexp(np.where(amax > 0, amax, 1.0))
    fl = exp - 1.0
    e = np.where(amax > 0, fl - E4M3_EMAX, -127.0)
    return np.clip(e, -127, 127).astype(np.int64)


def mx_quantize(v, block: int = BLOCK):
    """Quantize rows of v ([..., K], K a multiple of 32) per 32 values along
    the last axis.  Returns (codes uint8 [..., K], scales uint8 [..., K/32])."""
    v = np.asarray(v, np.float64)
    K = v.shape[-1]
    if K % block:
        raise ValueError("K must be a multiple of the block")
    vb = v.reshape(v.shape[:-1] + (K // block, block))
    amax = np.max(np.abs(vb), axis=-1)
    E = _block_exponent(amax)
    scaled = vb * np.exp2(-E.astype(np.float64))[..., None]
    codes = e4m3_encode(np.clip(scaled, -E4M3_MAX, E4M3_MAX)).reshape(v.shape)
    return codes, (E + 127).astype(np.uint8)


def mx_dequantize(codes, scales, block: int = BLOCK) -> np.ndarray:
    """float64 values of MX blocks: code value * 2^(scale - 127)."""
    c = np.asarray(codes, np.uint8)
    s = np.asarray(scales, np.uint8).astype(np.float64)
    vals = e4m3_decode(c)
    K = c.shape[-1]
    vb = vals.reshape(c.shape[:-1] + (K // block, block))
    return (vb * np.exp2(s - 127.0)[..., None]).reshape(c.shape)


def expert_ffn_mx(xq_vals, offsets, wgu_vals, wdn_vals):
    """Expert FFN on MX-quantized operands, in float64.

    xq_vals: [R, H] dequantized x_perm; wgu_vals [E_loc, 2I, H] and wdn_vals
    [E_loc, H, I] dequantized weights.  Returns (h64 [R, I] before
    quantization, h_codes, h_scales, y [R, H]) where y multiplies the
    dequantized h codes (h is GEMM2's MX operand)."""
    R = xq_vals.shape[0]
    E_loc, twoI, H = wgu_vals.shape
    I = twoI // 2
    h64 = np.zeros((R, I))
    for e in range(E_loc):
        a, b = int(offsets[e]), int(offsets[e + 1])
        if a == b:
            continue
        g = xq_vals[a:b] @ wgu_vals[e, :I].T
        u = xq_vals[a:b] @ wgu_vals[e, I:].T
        h64[a:b] = g / (1.0 + np.exp(-g)) * u
    h_codes, h_scales = mx_quantize(h64)
    hq = mx_dequantize(h_codes, h_scales)
    y = np.zeros((R, H))
    for e in range(E_loc):
        a, b = int(offsets[e]), int(offsets[e + 1])
        if a < b:
            y[a:b] = hq[a:b] @ wdn_vals[e].T
    return h64, h_codes, h_scales, y


def layer_mx(logits, x, wgu_codes, wgu_scales, wdn_codes, wdn_scales, k: int, e0: int):
    """The whole FP8 layer share: routing and layout as oracle/moe.py, x rows
    quantized to MX FP8, the expert FFN on MX operands, the float64 combine."""
    logits = np.asarray(logits)
    x = np.asarray(x, np.float64)
    T, H = x.shape
    E_loc = wgu_codes.shape[0]
    topk_idx, topk_w = moe.route(logits, k)
    le = moe.local_map(topk_idx, e0, E_loc)
    counts, offsets, row_of_slot, token_of_row = moe.layout(le, E_loc)
    xp = moe.permute(x, token_of_row)
    xp_codes, xp_scales = mx_quantize(xp)
    xq = mx_dequantize(xp_codes, xp_scales)
    wgu = mx_dequantize(wgu_codes, wgu_scales)
    wdn = mx_dequantize(wdn_codes, wdn_scales)
    h64, h_codes, h_scales, y = expert_ffn_mx(xq, offsets, wgu, wdn)
    out = moe.combine(y, topk_w, row_of_slot, T, H)
    return dict(topk_idx=topk_idx, topk_w=topk_w, counts=counts, offsets=offsets, row_of_slot=row_of_slot,
                token_of_row=token_of_row, x_codes=xp_codes, x_scales=xp_scales, h64=h64, h_codes=h_codes,
                h_scales=h_scales, y=y, out=out)
