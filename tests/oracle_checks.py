"""Pins for the CPU oracle: checks against things other than the oracle itself.

Each check takes a namespace `O` holding the oracle's stage functions
(route, local_map, layout, permute, expert_ffn, combine) and raises
AssertionError when the stage disagrees with a brute-force computation, a
closed form, a library routine or an invariant of the layer.  The pin tests
run them on the real oracle; the mutation test runs them on copies with a
planted mistake and expects each copy to fail at least one check.
"""

from __future__ import annotations

import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def compose_layer(O, logits, x, w_gu, w_dn, k, e0):
    T, H = x.shape
    idx, w = O.route(logits, k)
    le = O.local_map(idx, e0, w_gu.shape[0])
    counts, offsets, ros, tor = O.layout(le, w_gu.shape[0])
    xp = O.permute(x, tor)
    h, y = O.expert_ffn(xp, offsets, w_gu, w_dn)
    out = O.combine(y, w, ros, T, H)
    return dict(topk_idx=idx, topk_w=w, counts=counts, offsets=offsets, row_of_slot=ros, token_of_row=tor, h=h, y=y,
                out=out, x_perm=xp)


# ----------------------------------------------------------------------------- router


def check_router_bruteforce(O, seed=20):
    rng = np.random.default_rng(seed)
    for T, H, E in ((1, 1, 1), (3, 5, 2), (7, 64, 9), (4, 33, 17)):
        x = rng.standard_normal((T, H))
        w = rng.standard_normal((E, H))
        b = rng.standard_normal(E)
        for bias in (None, b):
            got = O.router_logits(x, w, bias)
            assert got.shape == (T, E)
            for t in range(T):
                for e in range(E):
                    ref = math.fsum(float(x[t, h]) * float(w[e, h]) for h in range(H))
                    if bias is not None:
                        ref += float(bias[e])
                    assert abs(got[t, e] - ref) <= 1e-12 * (1 + abs(ref)), (T, H, E, t, e)


def check_router_one_hot(O):
    # x = unit vectors pick columns of the gate matrix: logits[t] = w[:, h_t]
    H, E = 6, 4
    w = np.arange(E * H, dtype=np.float64).reshape(E, H) - 7.0
    x = np.zeros((H, H))
    x[np.arange(H), np.arange(H)] = 1.0
    assert np.array_equal(O.router_logits(x, w), w.T)
    assert np.array_equal(O.router_logits(x, w, np.full(E, 0.5)), w.T + 0.5)


# ----------------------------------------------------------------------------- route


def _brute_topk(row, k):
    # Python's own sort on (-value, id); -(-0.0) == -(+0.0) compare equal.
    order = sorted(range(len(row)), key=lambda e: (-float(row[e]), e))
    return order[:k]


def check_route_bruteforce(O, seed=0):
    rng = np.random.default_rng(seed)
    vals = np.array([-1.5, -0.0, 0.0, 0.75, 2.0, 3.25], np.float32)
    for E in (1, 2, 3, 5, 8, 13, 64, 70):
        for k in sorted({1, min(2, E), min(3, E), E}):
            T = 23
            logits = rng.choice(vals, size=(T, E)).astype(np.float32)
            idx, _ = O.route(logits, k)
            for t in range(T):
                assert list(idx[t]) == _brute_topk(logits[t], k), (E, k, t)
    # continuous values too
    logits = rng.standard_normal((40, 32)).astype(np.float32)
    idx, _ = O.route(logits, 4)
    for t in range(40):
        assert list(idx[t]) == _brute_topk(logits[t], 4)


def check_route_argmax(O, seed=1):
    rng = np.random.default_rng(seed)
    vals = np.array([-2.0, -0.0, 0.0, 1.0, 1.0], np.float32)
    logits = rng.choice(vals, size=(200, 9)).astype(np.float32)
    idx, w = O.route(logits, 1)
    # numpy's argmax returns the first maximum; -0.0 == +0.0 under '=='
    assert np.array_equal(idx[:, 0], np.argmax(logits, axis=1))
    assert np.all(w == 1.0)


def check_route_full_order(O, seed=2):
    rng = np.random.default_rng(seed)
    logits = rng.choice(np.array([-1.0, 0.0, -0.0, 2.0], np.float32), size=(50, 7)).astype(np.float32)
    idx, w = O.route(logits, 7)
    for t in range(50):
        assert sorted(idx[t]) == list(range(7))
        v = logits[t, idx[t]]
        assert np.all(v[:-1] >= v[1:])
        for j in range(6):
            if v[j] == v[j + 1]:
                assert idx[t, j] < idx[t, j + 1]
    # k = E: weights are the plain softmax of the token's logits, in slot order
    for t in range(50):
        z = [math.exp(float(l)) for l in logits[t]]
        s = sum(z)
        for j in range(7):
            assert abs(w[t, j] - z[idx[t, j]] / s) < 1e-12


def check_route_weights_closed_form(O, seed=3):
    rng = np.random.default_rng(seed)
    # renormalised softmax == softmax of the selected logits (written with math.exp)
    logits = (rng.standard_normal((60, 16)) * 3).astype(np.float32)
    idx, w = O.route(logits, 4)
    for t in range(60):
        z = [math.exp(float(logits[t, e])) for e in idx[t]]
        s = sum(z)
        for j in range(4):
            assert abs(w[t, j] - z[j] / s) < 1e-12
        assert abs(sum(w[t]) - 1.0) < 1e-12
    # E = k = 2: w0 = sigmoid(l_first - l_second)
    l2 = rng.standard_normal((30, 2)).astype(np.float32)
    idx, w = O.route(l2, 2)
    for t in range(30):
        a, b = float(l2[t, idx[t, 0]]), float(l2[t, idx[t, 1]])
        assert abs(w[t, 0] - 1.0 / (1.0 + math.exp(b - a))) < 1e-12
    # shift invariance of both selection and weights
    base = rng.standard_normal((20, 10)).astype(np.float32)
    shift = np.float32(0.5)
    i1, w1 = O.route(base, 3)
    i2, w2 = O.route(base + shift, 3)
    ok = np.all(np.argsort(-base, axis=1, kind="stable") == np.argsort(-(base + shift), axis=1, kind="stable"), axis=1)
    assert np.array_equal(i1[ok], i2[ok])
    assert np.allclose(w1[ok], w2[ok], rtol=0, atol=1e-6)


def check_route_golden(O):
    path = os.path.join(GOLDEN, "route_tiny.txt")
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        a, b, c = (p.split() for p in line.split("|"))
        logits = np.array([[float(v) for v in a]], np.float32)
        idx, w = O.route(logits, 2)
        assert list(idx[0]) == [int(v) for v in b], line
        assert np.allclose(w[0], [float(v) for v in c], rtol=0, atol=1e-6), (line, w)


# ----------------------------------------------------------------------------- layout


def _parse_pairs(s):
    return [[int(v) for v in grp.split()] for grp in s.split("|")]


def check_layout_golden(O):
    fields = {}
    for line in open(os.path.join(GOLDEN, "layout_tiny.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, val = line.split(":", 1)
        fields[key.strip()] = val.strip()
    le = np.array(_parse_pairs(fields["le"]), np.int32)
    counts, offsets, ros, tor = O.layout(le, 3)
    assert list(counts) == [int(v) for v in fields["counts"].split()]
    assert list(offsets) == [int(v) for v in fields["offsets"].split()]
    assert ros.tolist() == _parse_pairs(fields["row_of_slot"])
    assert list(tor) == [int(v) for v in fields["token_of_row"].split()]


def check_layout_library(O, seed=4):
    rng = np.random.default_rng(seed)
    for (T, k, E, E_loc, e0) in [(1, 1, 4, 4, 0), (37, 2, 8, 8, 0), (100, 4, 32, 32, 0), (257, 8, 256, 32, 64),
                                 (64, 3, 40, 5, 35), (0, 2, 8, 8, 0)]:
        logits = rng.standard_normal((T, E)).astype(np.float32)
        idx, _ = O.route(logits, k)
        le = O.local_map(idx, e0, E_loc)
        # local map against a per-element definition
        for t in range(T):
            for j in range(k):
                g = int(idx[t, j])
                assert le[t, j] == (g - e0 if e0 <= g < e0 + E_loc else -1)
        counts, offsets, ros, tor = O.layout(le, E_loc)
        flat = le.reshape(-1)
        kept = flat >= 0
        assert np.array_equal(counts, np.bincount(flat[kept], minlength=E_loc)[:E_loc])
        assert np.array_equal(offsets, np.concatenate([[0], np.cumsum(counts)]))
        assert counts.sum() + np.count_nonzero(~kept) == T * k
        # rows == positions of the kept slots in a stable sort by expert
        order = np.argsort(np.where(kept, flat, E_loc), kind="stable")[: int(kept.sum())]
        expect = np.full(T * k, -1, np.int64)
        expect[order] = np.arange(order.size)
        assert np.array_equal(ros.reshape(-1), expect)
        # every kept slot appears exactly once; tokens ascend within an expert
        assert np.array_equal(np.sort(ros.reshape(-1)[kept]), np.arange(int(kept.sum())))
        for e in range(E_loc):
            seg = tor[offsets[e]: offsets[e + 1]]
            assert np.all(np.diff(seg) > 0)
            for t in seg:
                assert e in le[t]
        assert np.array_equal(tor[expect[kept]], np.nonzero(kept)[0] // k)


# ----------------------------------------------------------------------------- ffn


def _brute_ffn_row(x, w_gu_e, w_dn_e, H, I):
    hh = []
    for i in range(I):
        g = sum(float(x[c]) * float(w_gu_e[i, c]) for c in range(H))
        u = sum(float(x[c]) * float(w_gu_e[I + i, c]) for c in range(H))
        hh.append(g / (1.0 + math.exp(-g)) * u)
    y = [sum(hh[i] * float(w_dn_e[o, i]) for i in range(I)) for o in range(H)]
    return hh, y


def check_ffn_bruteforce(O, seed=5):
    rng = np.random.default_rng(seed)
    E_loc, H, I = 3, 5, 3
    counts = [2, 0, 3]
    offsets = np.array([0, 2, 2, 5], np.int32)
    xp = rng.standard_normal((5, H)).astype(np.float32)
    w_gu = rng.standard_normal((E_loc, 2 * I, H)).astype(np.float32)
    w_dn = rng.standard_normal((E_loc, H, I)).astype(np.float32)
    h, y = O.expert_ffn(xp, offsets, w_gu, w_dn)
    for e in range(E_loc):
        for r in range(offsets[e], offsets[e + 1]):
            hh, yy = _brute_ffn_row(xp[r], w_gu[e], w_dn[e], H, I)
            assert np.allclose(h[r], hh, rtol=1e-12, atol=1e-12)
            assert np.allclose(y[r], yy, rtol=1e-12, atol=1e-12)
    assert counts[1] == 0


def check_dense_mlp(O, seed=6):
    """E = k = 1: the layer is a dense SwiGLU MLP applied to every token."""
    rng = np.random.default_rng(seed)
    T, H, I = 7, 6, 4
    x = rng.standard_normal((T, H)).astype(np.float32)
    w_gu = rng.standard_normal((1, 2 * I, H)).astype(np.float32)
    w_dn = rng.standard_normal((1, H, I)).astype(np.float32)
    logits = rng.standard_normal((T, 1)).astype(np.float32)
    res = compose_layer(O, logits, x, w_gu, w_dn, 1, 0)
    for t in range(T):
        _, yy = _brute_ffn_row(x[t], w_gu[0], w_dn[0], H, I)
        assert np.allclose(res["out"][t], yy, rtol=1e-12, atol=1e-12)


# ----------------------------------------------------------------------------- combine / whole layer


def check_identity_experts(O, seed=7):
    """y := x_perm gives out = (sum of resident weights) * x, = x if all resident."""
    rng = np.random.default_rng(seed)
    for (T, k, E, E_loc, e0) in [(33, 4, 16, 16, 0), (40, 2, 8, 8, 0), (50, 3, 12, 5, 4), (20, 1, 6, 6, 0)]:
        logits = rng.standard_normal((T, E)).astype(np.float32)
        x = rng.standard_normal((T, 6)).astype(np.float32)
        idx, w = O.route(logits, k)
        le = O.local_map(idx, e0, E_loc)
        counts, offsets, ros, tor = O.layout(le, E_loc)
        xp = O.permute(x, tor)
        assert np.array_equal(xp, x[tor])
        out = O.combine(xp.astype(np.float64), w, ros, T, 6)
        wsum = np.where(le >= 0, w, 0.0).sum(axis=1)
        assert np.allclose(out, wsum[:, None] * x, rtol=1e-12, atol=1e-12)
        if E_loc == E:
            assert np.allclose(out, x, rtol=1e-12, atol=1e-12)
        if k == 1:
            assert np.array_equal(out, x.astype(np.float64))


def check_ep_shares_sum(O, seed=8):
    """Summing the shares of all GPUs of an expert-parallel group gives the
    layer computed with every expert resident."""
    rng = np.random.default_rng(seed)
    T, E, k, H, I, G = 19, 12, 3, 6, 4, 4
    x = rng.standard_normal((T, H)).astype(np.float32)
    logits = rng.standard_normal((T, E)).astype(np.float32)
    w_gu = rng.standard_normal((E, 2 * I, H)).astype(np.float32)
    w_dn = rng.standard_normal((E, H, I)).astype(np.float32)
    full = compose_layer(O, logits, x, w_gu, w_dn, k, 0)["out"]
    per = E // G
    acc = np.zeros_like(full)
    for g in range(G):
        sl = slice(g * per, (g + 1) * per)
        acc += compose_layer(O, logits, x, w_gu[sl], w_dn[sl], k, g * per)["out"]
    assert np.allclose(acc, full, rtol=1e-12, atol=1e-12)
    # and against a per-token brute force of the full layer
    for t in range(T):
        order = _brute_topk(logits[t], k)
        z = [math.exp(float(logits[t, e])) for e in order]
        s = sum(z)
        ref = np.zeros(H)
        for j, e in enumerate(order):
            _, yy = _brute_ffn_row(x[t], w_gu[e], w_dn[e], H, I)
            ref += (z[j] / s) * np.array(yy)
        assert np.allclose(full[t], ref, rtol=1e-10, atol=1e-10)


def check_permute_slots(O, seed=9):
    """Permute against its definition from the slot side: every resident
    (token, slot) pair owns one row, whose x_perm row is that token's hidden
    row, and no row is left over (each (token, slot) appears exactly once)."""
    rng = np.random.default_rng(seed)
    for (T, k, E, E_loc, e0) in [(1, 1, 3, 3, 0), (29, 3, 10, 10, 0), (64, 4, 16, 6, 5), (40, 8, 64, 32, 32)]:
        logits = rng.standard_normal((T, E)).astype(np.float32)
        x = rng.standard_normal((T, 5)).astype(np.float32)
        idx, _ = O.route(logits, k)
        le = O.local_map(idx, e0, E_loc)
        counts, offsets, ros, tor = O.layout(le, E_loc)
        xp = O.permute(x, tor)
        R = int(offsets[-1])
        assert xp.shape == (R, 5)
        seen = np.zeros(R, np.int64)
        for t in range(T):
            for j in range(k):
                r = int(ros[t, j])
                if le[t, j] < 0:
                    assert r == -1
                    continue
                seen[r] += 1
                for h in range(5):
                    assert xp[r, h] == x[t, h], (T, t, j, r)
        assert np.all(seen == 1)


ALL_CHECKS = [
    check_router_bruteforce,
    check_router_one_hot,
    check_route_bruteforce,
    check_route_argmax,
    check_route_full_order,
    check_route_weights_closed_form,
    check_route_golden,
    check_layout_golden,
    check_layout_library,
    check_ffn_bruteforce,
    check_dense_mlp,
    check_identity_experts,
    check_permute_slots,
    check_ep_shares_sum,
]
