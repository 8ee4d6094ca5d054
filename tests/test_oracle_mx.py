"""Pins of the MX FP8 oracle (oracle/mx.py) against things other than itself:
PyTorch's float8_e4m3fn conversions (a library routine implementing the OCP
E4M3 format), a brute-force nearest-code search, hand-worked blocks, error
bounds of the format, and a scalar per-token re-implementation of the FP8
layer."""

import math

import numpy as np
import pytest

from oracle import moe
from oracle import mx


def _finite_codes():
    return [c for c in range(256) if (c & 0x7F) != 0x7F]


def test_decode_matches_torch_float8():
    torch = pytest.importorskip("torch")
    c = np.arange(256, dtype=np.uint8)
    got = mx.e4m3_decode(c)
    ref = torch.from_numpy(c.copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan) and nan.sum() == 2
    assert np.array_equal(got[~nan], ref[~nan])
    assert mx.e4m3_decode(0x7E) == 448 and mx.e4m3_decode(0x01) == 2.0 ** -9 and mx.e4m3_decode(0x08) == 2.0 ** -6


def _midpoints():
    pos = sorted({float(mx.e4m3_decode(c)) for c in _finite_codes() if c < 0x80})
    out = []
    for a, b in zip(pos, pos[1:]):
        m = 0.5 * (a + b)
        out += [m, math.nextafter(m, 0.0), math.nextafter(m, 1e9)]
    out += pos
    return np.array(out + [-v for v in out] + [0.0, -0.0])


def test_encode_matches_torch_in_range():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(1)
    v = np.concatenate([_midpoints(), rng.standard_normal(20000) * 40, rng.standard_normal(5000) * 0.01])
    v = v[np.abs(v) <= 448].astype(np.float32)  # torch does not saturate; in range only
    ref = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(mx.e4m3_encode(v), ref)


def test_encode_is_the_nearest_code_ties_to_even():
    vals = {c: float(mx.e4m3_decode(c)) for c in _finite_codes()}
    for v in _midpoints():
        best = None
        for c, d in vals.items():
            if d == 0 and math.copysign(1, v) != (-1 if c & 0x80 else 1):
                continue  # a zero result keeps the sign
            key = (abs(d - v), c & 1)  # nearer first, then the even mantissa
            if best is None or key < best[0]:
                best = (key, c)
        assert int(mx.e4m3_encode(v)) == best[1], v


def test_encode_saturates():
    assert list(mx.e4m3_encode([448.0, 449.0, 1e6, -500.0, -448.0])) == [0x7E, 0x7E, 0x7E, 0xFE, 0xFE]


def test_quantize_hand_worked_blocks():
    # amax 3 -> E = floor(log2 3) - 8 = -7 (scale byte 120); 3 * 2^7 = 384 =
    # 1.5 * 2^8 -> code 0x7C; 0.5 * 2^7 = 64 = 2^6 -> code (13 << 3) = 104
    c, s = mx.mx_quantize(np.array([[3.0] + [0.5] * 31]))
    assert s.tolist() == [[120]] and c[0, 0] == 0x7C and (c[0, 1:] == 104).all()
    # amax 3.9: 3.9 * 128 = 499.2 clips to 448 (dequantized 3.5)
    c, s = mx.mx_quantize(np.array([[3.9] + [0.0] * 31]))
    assert s[0, 0] == 120 and c[0, 0] == 0x7E and mx.mx_dequantize(c, s)[0, 0] == 3.5
    # a power-of-two maximum lands on 256 exactly
    c, s = mx.mx_quantize(np.array([[-2.0 ** -20] + [2.0 ** -30] * 31]))
    assert s[0, 0] == 127 - 28 and c[0, 0] == 0x80 | (15 << 3) and mx.mx_dequantize(c, s)[0, 0] == -2.0 ** -20
    # an all-zero block: scale 2^-127 and zero codes (signs kept)
    c, s = mx.mx_quantize(np.array([[0.0, -0.0] * 16]))
    assert s[0, 0] == 0 and c[0, 0] == 0x00 and c[0, 1] == 0x80
    # two blocks per row are independent
    c, s = mx.mx_quantize(np.array([[1.0] * 32 + [8.0] * 32]))
    assert s.tolist() == [[127 - 8, 127 - 5]]


def test_quantize_error_bound():
    rng = np.random.default_rng(2)
    v = rng.standard_normal((64, 256)) * np.exp2(rng.integers(-12, 12, size=(64, 1)))
    c, s = mx.mx_quantize(v)
    d = mx.mx_dequantize(c, s)
    E = s.astype(np.float64) - 127
    step = np.repeat(np.exp2(E), 32, axis=1)
    scaled = np.abs(v) / step
    # half an E4M3 ulp at each value (2^-4 relative for normals, 2^-10 below
    # 2^-6), or the clip to 448
    half = np.where(scaled >= 2.0 ** -6, np.exp2(np.floor(np.log2(np.maximum(scaled, 1e-300))) - 4), 2.0 ** -10)
    bound = np.where(scaled > 448, scaled - 448, half) * step
    assert (np.abs(d - v) <= bound * (1 + 1e-12)).all()
    # the block maximum lands in [256, 512) before the clip
    bmax = np.max(np.abs(v).reshape(64, 8, 32), axis=2) / np.exp2(s - 127.0)
    assert ((bmax >= 256) & (bmax < 512)).all()


# ---------------------------------------------------------------- layer, scalar re-implementation


def _q_scalar(vals):
    """One block by the rule, value by value with the math module."""
    amax = max(abs(v) for v in vals)
    E = math.frexp(amax)[1] - 1 - 8 if amax > 0 else -127
    E = max(-127, min(127, E))
    out = []
    for v in vals:
        a = min(abs(v) * 2.0 ** -E, 448.0)
        if a < 2.0 ** -6:
            q = round(a * 512) / 512  # Python rounds half to even
        else:
            e = math.frexp(a)[1] - 1
            q = round(a / 2.0 ** e * 8) / 8 * 2.0 ** e
        out.append(math.copysign(q, v) * 2.0 ** E)
    return out


def _q_row(row):
    out = []
    for b in range(0, len(row), 32):
        out += _q_scalar(row[b:b + 32])
    return out


def test_layer_against_scalar_per_token_loops():
    rng = np.random.default_rng(3)
    T, E, k, H, I, e0, E_loc = 9, 6, 2, 64, 32, 1, 4
    logits = rng.standard_normal((T, E)).astype(np.float32)
    x = rng.standard_normal((T, H))
    wgu_c, wgu_s = mx.mx_quantize(rng.standard_normal((E_loc, 2 * I, H)) * 0.2)
    wdn_c, wdn_s = mx.mx_quantize(rng.standard_normal((E_loc, H, I)) * 0.2)
    res = mx.layer_mx(logits, x, wgu_c, wgu_s, wdn_c, wdn_s, k, e0)
    wgu = mx.mx_dequantize(wgu_c, wgu_s)
    wdn = mx.mx_dequantize(wdn_c, wdn_s)
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-float(logits[t, e]), e))[:k]
        z = [math.exp(float(logits[t, e])) for e in order]
        xq = _q_row([float(v) for v in x[t]])
        acc = [0.0] * H
        for j, e in enumerate(order):
            le = e - e0
            if not (0 <= le < E_loc):
                continue
            g = [math.fsum(xq[c] * wgu[le, i, c] for c in range(H)) for i in range(I)]
            u = [math.fsum(xq[c] * wgu[le, I + i, c] for c in range(H)) for i in range(I)]
            h = _q_row([g[i] / (1 + math.exp(-g[i])) * u[i] for i in range(I)])
            w = z[j] / sum(z)
            for c in range(H):
                acc[c] += w * math.fsum(h[i] * wdn[le, c, i] for i in range(I))
        assert np.allclose(res["out"][t], acc, rtol=1e-9, atol=1e-12), t
