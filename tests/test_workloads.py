"""CPU checks of the synthetic workloads (inputs only, no GPU)."""
import numpy as np

import oracle
from synth import CONFIGS
from synth.gen import _draw_block, _stream, seed_of, stored_bias


def test_skewed_bias_reaches_capped_zipf_shares():
    """Config 3's stored router bias, on fresh tokens (not the calibration
    set), gives slot shares close to the target min(1/8, c r^-1.2): the two
    head experts at the 1/8 cap, the resident block [0, 32) near 74.8 %, and
    popularity falling with the expert id."""
    spec = CONFIGS[3]
    seed = seed_of(3)
    b = stored_bias(3).astype(np.float64)
    wg = _stream(seed, 0).standard_normal(size=(spec.H, spec.E), dtype=np.float32) * np.float32(1 / np.sqrt(spec.H))
    x, _ = _draw_block(seed, (1 << 20) + 7, (2048, spec.H), 1.0, spec.dtype)
    logits = (x.astype(np.float64) @ wg.astype(np.float64) + b[None, :]).astype(np.float32)
    idx, _ = oracle.route(logits, spec.k)
    f = np.bincount(idx.ravel(), minlength=spec.E) / idx.size
    r = np.arange(1, spec.E + 1, dtype=np.float64)
    assert abs(f[0] - 1 / 8) < 0.01 and abs(f[1] - 1 / 8) < 0.01
    resident = f[:spec.E_loc].sum()
    assert abs(resident - 0.748) < 0.03, resident
    # shares of ranks 3..32 within 25 % of c r^-1.2 (c from the cap-free tail)
    c = 0.08 * 3 ** 1.2
    rel = f[2:32] / (c * r[2:32] ** -1.2)
    assert np.all(np.abs(rel - 1) < 0.25), rel
    # popularity decreases in blocks of eight ids
    blocks = f[:64].reshape(8, 8).sum(axis=1)
    assert np.all(np.diff(blocks) < 0)


def test_uniform_configs_have_no_bias():
    for cfg in (0, 1, 2):
        assert CONFIGS[cfg].zipf_s is None


def test_agentic_trace_matches_its_recipe():
    """The agentic trace: 200 seeded steps, D batches uniform on 32..256, a P
    batch on about half the steps with log-uniform size on 512..16384, and
    every batch a window inside its token pool."""
    import math

    from synth import agentic_trace

    tr = agentic_trace()
    assert len(tr) == 200 and tr == agentic_trace()  # deterministic
    td = np.array([s.t_d for s in tr])
    tp = np.array([s.t_p for s in tr if s.t_p])
    assert td.min() >= 32 and td.max() <= 256 and abs(td.mean() - 144) < 15
    assert 70 <= len(tp) <= 130
    assert tp.min() >= 512 and tp.max() <= 16384
    # log-uniform: log(size) roughly uniform on [log 512, log 16384]
    u = (np.log(tp) - math.log(512)) / (math.log(16384) - math.log(512))
    assert abs(u.mean() - 0.5) < 0.1
    for s in tr:
        assert 0 <= s.d_off and s.d_off + s.t_d <= 256
        assert 0 <= s.p_off and s.p_off + s.t_p <= 16384
