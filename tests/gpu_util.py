"""Helpers for the GPU tests: upload seeded inputs, drive the C ABI through
the binding, read the phase-owned buffers back, compare with the oracle."""

from __future__ import annotations

import ctypes
import math

import numpy as np

from synth import BF16, FP8, bf16_bits_to_f32

_hip = None


def hip():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        _hip.hipMemcpy.restype = ctypes.c_int
    return _hip


def hip_last_error() -> str:
    h = hip()
    h.hipGetLastError.restype = ctypes.c_int
    h.hipGetErrorString.restype = ctypes.c_char_p
    h.hipGetErrorString.argtypes = [ctypes.c_int]
    e = h.hipGetLastError()
    return f"{e} ({h.hipGetErrorString(e).decode()})"


def read_dev(ptr: int, shape, dtype) -> np.ndarray:
    """Copy device memory at `ptr` into a new host array (after a device sync)."""
    a = np.empty(shape, dtype)
    if a.nbytes == 0:
        return a
    st = hip().hipMemcpy(a.ctypes.data, ptr, a.nbytes, 2)  # device to host
    assert st == 0, f"hipMemcpy failed ({st})"
    return a


def to_dev(a: np.ndarray):
    import torch

    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        t = torch.from_numpy(a.view(np.int16))
    else:
        t = torch.from_numpy(a)
    return t.to("cuda")


class GpuLayer:
    """One context over a LayerInputs, with per-phase streams and outputs."""

    def __init__(self, inp, max_tokens=None, d_priority_us=0):
        import torch

        from paper_2609_00993_amd import moepd as M

        self.M = M
        self.inp = inp
        spec = inp.spec
        self.spec = spec
        self.bf16 = spec.dtype == BF16
        self.fp8 = spec.dtype == FP8
        self.T = {0: spec.T_P, 1: spec.T_D}
        if max_tokens is None:
            max_tokens = (spec.T_P, spec.T_D)
        packed = self.bf16 or self.fp8  # weights as bit patterns / codes
        self.w_gu = to_dev(inp.w_gu_bits if packed else inp.w_gu)
        self.w_dn = to_dev(inp.w_dn_bits if packed else inp.w_dn)
        self.w_gu_s = to_dev(inp.w_gu_scales) if self.fp8 else None
        self.w_dn_s = to_dev(inp.w_dn_scales) if self.fp8 else None
        self.x = {ph: to_dev(inp.x_bits[ph] if packed else inp.x[ph]) for ph in (0, 1)}
        self.logits = {ph: to_dev(inp.logits[ph]) for ph in (0, 1)}
        self.out = {ph: torch.zeros((self.T[ph], spec.H), dtype=torch.float32, device="cuda") for ph in (0, 1)}
        torch.cuda.synchronize()  # the fills run on torch's stream, which ours do not wait for
        dt = M.MOE_DTYPE_FP8 if self.fp8 else M.MOE_DTYPE_BF16 if self.bf16 else M.MOE_DTYPE_F32
        cfg = M.make_config(spec.E, spec.e0, spec.E_loc, spec.k, spec.H, spec.I, dt, max_tokens[0], max_tokens[1],
                            d_priority_us=d_priority_us)
        st, self.ctx = M.moe_ctx_create(cfg, self.w_gu, self.w_dn, self.w_gu_s, self.w_dn_s)
        if st == M.MOE_ERR_HIP:
            err = hip_last_error()
            raise AssertionError(f"moe_ctx_create: HIP error {err} (free/total {torch.cuda.mem_get_info()})")
        M.check(st, "moe_ctx_create")
        self.streams = {0: torch.cuda.Stream(), 1: torch.cuda.Stream()}

    def run(self, ph, stream=None, T=None):
        T = self.T[ph] if T is None else T
        s = self.streams[ph] if stream is None else stream
        self.M.layer(self.ctx, ph, self.logits[ph], T, self.x[ph], self.out[ph], s)

    def fetch(self, ph):
        import torch

        torch.cuda.synchronize()
        M, spec = self.M, self.spec
        st, v = M.moe_phase_view(self.ctx, ph)
        M.check(st)
        T, k = v.tokens, spec.k
        res = dict(
            topk_idx=read_dev(v.topk_idx, (T, k), np.int32),
            topk_w=read_dev(v.topk_w, (T, k), np.float32),
            counts=read_dev(v.counts, (spec.E_loc,), np.int32),
            offsets=read_dev(v.offsets, (spec.E_loc + 1,), np.int32),
            row_of_slot=read_dev(v.row_of_slot, (T, k), np.int32),
        )
        R = int(res["offsets"][-1])
        res["R"] = R
        res["token_of_row"] = read_dev(v.token_of_row, (R,), np.int32)
        res["y"] = read_dev(v.y, (R, spec.H), np.float32)
        res["out"] = self.out[ph].cpu().numpy()
        if self.fp8:
            res["x_codes"] = read_dev(v.x_perm, (R, spec.H), np.uint8)
            res["x_scales"] = read_dev(v.x_perm_scales, (R, spec.H // 32), np.uint8)
            res["h_codes"] = read_dev(v.h, (R, spec.I), np.uint8)
            res["h_scales"] = read_dev(v.h_scales, (R, spec.I // 32), np.uint8)
            return res
        edt = np.uint16 if self.bf16 else np.float32
        res["x_perm_raw"] = read_dev(v.x_perm, (R, spec.H), edt)
        res["h_raw"] = read_dev(v.h, (R, spec.I), edt)
        for key in ("x_perm", "h"):
            raw = res[key + "_raw"]
            res[key] = bf16_bits_to_f32(raw) if self.bf16 else raw
        return res

    def close(self):
        if self.ctx:
            self.M.check(self.M.moe_ctx_destroy(self.ctx))
            self.ctx = None


def rms(a) -> float:
    a = np.asarray(a, np.float64)
    return math.sqrt(float(np.mean(a * a))) if a.size else 0.0


def tol_of(spec) -> float:
    """Max |gpu - oracle| allowed on the layer output, as a fraction of the
    oracle output's RMS: 2e-2 for bf16 layers, 1e-5 for float32 layers."""
    return 2e-2 if spec.dtype == BF16 else 1e-5


# Intermediate tensors have heavy tails (h = silu(g) u reaches ~20x its RMS),
# so they are checked element by element against the precision they are
# stored in rather than against the output's RMS bar:
#  * bf16 h = RNE(h32): |h - h_ref| <= 2^-8 |h_ref| (half a bf16 ulp is at most
#    2^-8 relative) + a floor of 1e-3 RMS for the float32 accumulation of g, u;
#  * float32 y = h_bf16 W2^T: each h_i carries <= 2^-8 |h_i| error, so
#    |y - y_ref| <= 2^-8 (|h_ref| |W2|^T) + 1e-3 RMS(y_ref);
#  * float32 layers: |err| <= 1e-5 (|ref| + RMS(ref)) for h and y (float32
#    accumulation over K <= 512 products, tails included).
BF16_REL = 2.0 ** -8


def assert_elementwise(got, ref, bound, what=""):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if ref.size == 0:
        return
    err = np.abs(got - ref)
    bad = err > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} elements over the bound; worst excess "
                           f"{float(np.max(err - bound)):.3e}")


def check_h_y(res, ref, w_dn, offsets, spec, what=""):
    """Check h and y of the GPU against the oracle's, element by element."""
    h, y = res["h"], res["y"]
    h_ref, y_ref = ref["h"], ref["y"]
    if spec.dtype == BF16:
        assert_elementwise(h, h_ref, BF16_REL * np.abs(h_ref) + 1e-3 * rms(h_ref), f"{what} h")
        cond = np.zeros_like(y_ref)
        ah = np.abs(h_ref)
        for e in range(len(offsets) - 1):
            a, b = int(offsets[e]), int(offsets[e + 1])
            if a < b:
                cond[a:b] = ah[a:b] @ np.abs(np.asarray(w_dn[e], np.float64)).T
        assert_elementwise(y, y_ref, BF16_REL * cond + 1e-3 * rms(y_ref), f"{what} y")
    else:
        assert_elementwise(h, h_ref, 1e-5 * (np.abs(h_ref) + rms(h_ref)), f"{what} h")
        assert_elementwise(y, y_ref, 1e-5 * (np.abs(y_ref) + rms(y_ref)), f"{what} y")


# float32 gate weights: l_j - l_0 rounds (|diff| < 16 -> <= 1e-6 relative after
# exp), expf and the k-term sum and divide add a few ulp: 2e-6 relative.
W_RTOL = 2e-6


def assert_route_layout_exact(res, ref, what=""):
    assert np.array_equal(res["topk_idx"], ref["topk_idx"]), f"{what} topk_idx"
    w, rw = res["topk_w"].astype(np.float64), ref["topk_w"]
    err = np.abs(w - rw) / np.maximum(np.abs(rw), 1e-30)
    assert err.size == 0 or err.max() <= W_RTOL, f"{what} topk_w rel err {err.max()}"
    for key in ("counts", "offsets", "row_of_slot", "token_of_row"):
        assert np.array_equal(res[key], ref[key]), f"{what} {key}"


def assert_close_rms(got, ref, tol, what=""):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if ref.size == 0:
        return
    scale = rms(ref)
    err = float(np.max(np.abs(got - ref)))
    assert err <= tol * scale, f"{what}: max|err| {err:.3e} > {tol:g} x rms {scale:.3e}"


def covering_rows(offsets, stride: int = 32) -> np.ndarray:
    """Rows that cover every m-tile of every expert segment: each segment's
    first row, every stride-th row after it, the row just before each of
    those, and its last row.  Any tile of at least `stride` rows that starts
    at a segment's start or at a multiple of at least `stride` rows into it
    (all the GEMMs' tile shapes: 32-row decode tiles, 160-row tiles with the
    rows shared evenly, 256-row tiles) holds one of them, and so does each
    expert's ragged tail.  Sorted, so the rows stay grouped by expert."""
    off = np.asarray(offsets, np.int64)
    rows = []
    for e in range(len(off) - 1):
        a, b = int(off[e]), int(off[e + 1])
        if a == b:
            continue
        r = np.arange(a, b, stride)
        rows.append(r)
        rows.append(np.maximum(r - 1, a))
        rows.append(np.minimum(r + stride - 1, b - 1))
        rows.append(np.array([b - 1]))
    if not rows:
        return np.zeros(0, np.int64)
    return np.unique(np.concatenate(rows))


def sub_offsets(rows, offsets) -> np.ndarray:
    """Offsets of the experts' segments within a sorted subset of rows."""
    return np.searchsorted(np.asarray(rows), np.asarray(offsets, np.int64)).astype(np.int64)


def check_rows_h_y(res, inp, ph, rows, offsets, token_of_row, what=""):
    """h and y of a subset of rows (sorted, so grouped by expert) against the
    oracle's expert FFN on the same rows, element by element (check_h_y's
    bounds).  A row's h and y depend only on its own x row and expert."""
    import oracle

    spec = inp.spec
    so = sub_offsets(rows, offsets)
    xr = inp.x[ph][np.asarray(token_of_row)[rows]]
    h_ref, y_ref = oracle.expert_ffn(xr, so, inp.w_gu, inp.w_dn)
    got = dict(h=res["h"][rows], y=res["y"][rows])
    check_h_y(got, dict(h=h_ref, y=y_ref), inp.w_dn, so, spec, what)


def sample_tokens(T: int, row_tokens, n_uniform: int, n_rows: int, seed: int):
    """A seeded uniform sample of tokens (its output RMS stands for the whole
    phase's) and a seeded sample of the tokens that own covering rows."""
    rng = np.random.default_rng(seed)
    uni = np.sort(rng.choice(T, size=min(T, n_uniform), replace=False))
    own = np.unique(np.asarray(row_tokens))
    if own.size > n_rows:
        own = np.sort(rng.choice(own, size=n_rows, replace=False))
    return uni, own


def check_out_sampled(res, inp, ph, uni, own, tol, what=""):
    """The layer output of sampled tokens against the oracle run on the
    sampled sub-batch (a token's output depends on no other token).  The bar
    is tol x the RMS of the oracle's output over the uniform sample, an
    unbiased stand-in for the RMS over the whole phase batch."""
    import oracle

    spec = inp.spec
    toks = np.union1d(uni, own)
    sub = oracle.layer(inp.logits[ph][toks], inp.x[ph][toks], inp.w_gu, inp.w_dn, spec.k, spec.e0)
    scale = rms(sub["out"][np.searchsorted(toks, uni)])
    got = np.asarray(res["out"][toks], np.float64)
    err = float(np.max(np.abs(got - sub["out"]))) if toks.size else 0.0
    assert err <= tol * scale, f"{what}: max|err| {err:.3e} > {tol:g} x rms {scale:.3e} ({toks.size} tokens)"
    return err / scale if scale else 0.0
