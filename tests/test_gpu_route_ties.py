"""GPU top-k on tied logits and signed zeros, through the C ABI.

Random continuous logits practically never tie, so the tie rule (equal
logits go to the lower expert id, -0.0 equals +0.0; the paper states top-8
routing, Section 7.1, and leaves ties open) is exercised here on logits drawn
from a few discrete levels that include both zeros, with planted runs of
+0.0 / -0.0 at the top of a row.  topk_idx must equal the oracle's exactly
and topk_w within the usual 2e-6 relative bound, over pool sizes on both
sides of the kernel's 64-experts-per-lane steps and every k up to 16."""

import numpy as np
import pytest

import oracle
from synth import tie_logits
from tests.gpu_util import W_RTOL, read_dev, to_dev

pytestmark = pytest.mark.gpu

CASES = [(E, k) for E in (8, 64, 65, 256, 300, 1024) for k in (1, 2, 8, 16) if k <= E]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def tied_batch(E, T, seed):
    rng = np.random.default_rng(seed)
    lg = np.concatenate([tie_logits(rng, T // 2, E, levels=7), tie_logits(rng, T - T // 2, E, levels=3)])
    # planted rows: every logit a signed zero, or a block of signed zeros
    # above a floor of negatives
    lg[0] = np.where(rng.random(E) < 0.5, np.float32(-0.0), np.float32(0.0))
    lg[1] = -1.0
    lg[1, E // 3:] = np.where(rng.random(E - E // 3) < 0.5, np.float32(-0.0), np.float32(0.0))
    lg[2] = np.float32(0.0)
    lg[2, ::2] = np.float32(-0.0)
    return lg.astype(np.float32)


@pytest.mark.parametrize("E,k", CASES)
def test_route_ties_exact(E, k):
    import torch

    from paper_2609_00993_amd import moepd as M

    T = {0: 1000, 1: 37}
    e_loc = min(E, 16)
    w_gu = torch.zeros((e_loc, 128, 64), dtype=torch.int16, device="cuda")
    w_dn = torch.zeros((e_loc, 64, 64), dtype=torch.int16, device="cuda")
    cfg = M.make_config(E, 0, e_loc, k, 64, 64, M.MOE_DTYPE_BF16, T[0], T[1])
    st, ctx = M.moe_ctx_create(cfg, w_gu, w_dn)
    M.check(st, "moe_ctx_create")
    try:
        s = torch.cuda.Stream()
        for ph in (0, 1):
            lg = tied_batch(E, T[ph], seed=E * 100 + k * 10 + ph)
            d = to_dev(lg)
            torch.cuda.synchronize()
            M.check(M.moe_route(ctx, ph, d, T[ph], s))
            torch.cuda.synchronize()
            st, v = M.moe_phase_view(ctx, ph)
            M.check(st)
            idx = read_dev(v.topk_idx, (T[ph], k), np.int32)
            w = read_dev(v.topk_w, (T[ph], k), np.float32).astype(np.float64)
            ridx, rw = oracle.route(lg, k)
            bad = np.nonzero(np.any(idx != ridx, axis=1))[0]
            assert bad.size == 0, (f"E={E} k={k} phase {ph}: {bad.size} rows differ, first {bad[0]}: "
                                   f"gpu {idx[bad[0]]} oracle {ridx[bad[0]]}")
            err = np.abs(w - rw) / np.maximum(np.abs(rw), 1e-30)
            assert err.max() <= W_RTOL, (E, k, ph, float(err.max()))
            M.check(M.moe_phase_reset(ctx, ph))
    finally:
        M.check(M.moe_ctx_destroy(ctx))
