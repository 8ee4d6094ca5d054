#!/usr/bin/env python3
"""Write tests/golden/zipf_bias_cfg3.txt: the per-expert router bias of the
skewed-routing workload (E = 256, top-8, H = 7168).

The workload asks for expert popularity that follows Zipf(s = 1.2).  Taken
literally that cannot hold at the head: with top-8 selection without
replacement no expert can receive more than 1/8 of all slots, and the Zipf
head would need about a quarter.  Reading used: target slot shares
p_r = min(1/8, c r^-1.2) over popularity rank r = expert id + 1, with c set
so that the shares sum to one (water filling), so the resident block
[0, 32) holds the head.

Calibration (seeded, deterministic): start from b = ln p; for 60 rounds,
route 4096 calibration tokens with the CPU oracle's top-k on the logits
x W_g + b, measure each expert's slot share f, and move b <- b + 0.5 ln(p / f)
(f floored at half a slot).  The calibration tokens are their own seeded
block of bf16-rounded normals; W_g is the workload's own router weight.

Only the oracle and the input generator are used, so the stored bias does not
depend on the GPU path.  Run from the repository root:
    python tests/golden/make_zipf_bias.py
"""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from synth.gen import CONFIGS, _draw_block, _stream, seed_of  # noqa: E402

OUT = os.path.join(ROOT, "tests", "golden", "zipf_bias_cfg3.txt")
CAL_TOKENS = 4096
ROUNDS = 60
CAL_BLOCK = 1 << 20  # seed block id of the calibration tokens (clear of the workload's blocks)


def target_shares(E: int, k: int, s: float) -> np.ndarray:
    """p_r = min(1/k, c r^-s), sum 1 (bisection on c)."""
    r = np.arange(1, E + 1, dtype=np.float64)
    lo, hi = 0.0, 1.0
    for _ in range(200):
        c = 0.5 * (lo + hi)
        tot = np.minimum(1.0 / k, c * r ** -s).sum()
        if tot < 1.0:
            lo = c
        else:
            hi = c
    p = np.minimum(1.0 / k, hi * r ** -s)
    return p / p.sum()


def main():
    spec = CONFIGS[3]
    seed = seed_of(3)
    E, k, H = spec.E, spec.k, spec.H
    p = target_shares(E, k, spec.zipf_s)
    wg = _stream(seed, 0).standard_normal(size=(H, E), dtype=np.float32) * np.float32(1.0 / np.sqrt(H))
    x_cal, _ = _draw_block(seed, CAL_BLOCK, (CAL_TOKENS, H), 1.0, spec.dtype)
    base = x_cal.astype(np.float64) @ wg.astype(np.float64)
    b = np.log(p)
    slots = CAL_TOKENS * k
    for _ in range(ROUNDS):
        idx, _ = oracle.route((base + b[None, :]).astype(np.float32), k)
        f = np.bincount(idx.ravel(), minlength=E) / slots
        b = b + 0.5 * np.log(p / np.maximum(f, 0.5 / slots))
    b32 = b.astype(np.float32)
    idx, _ = oracle.route((base + b32.astype(np.float64)[None, :]).astype(np.float32), k)
    f = np.bincount(idx.ravel(), minlength=E) / slots
    resident = f[spec.e0:spec.e0 + spec.E_loc].sum()
    with open(OUT, "w") as fh:
        fh.write("# Router bias of the skewed-routing workload (E=256, top-8, H=7168), one float32 per expert id.\n")
        fh.write("# Written by tests/golden/make_zipf_bias.py (oracle top-k calibration; see its docstring).\n")
        fh.write(f"# calibration tokens {CAL_TOKENS}, rounds {ROUNDS}; realised resident share {resident:.4f} "
                 f"(target {p[spec.e0:spec.e0 + spec.E_loc].sum():.4f}); head shares "
                 + " ".join(f"{v:.4f}" for v in f[:4]) + " (target " + " ".join(f"{v:.4f}" for v in p[:4]) + ")\n")
        for v in b32:
            fh.write(f"{float(v):.9g}\n")
    print(f"wrote {OUT}: resident share {resident:.4f}, max share {f.max():.4f}")


if __name__ == "__main__":
    main()
