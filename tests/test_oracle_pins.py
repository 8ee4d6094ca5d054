"""The CPU oracle against its pins (brute force, closed forms, library
routines, invariants, hand-computed fixtures), plus a mutation test showing
that each plausible mistake planted in a copy of the oracle fails a pin."""

import types

import numpy as np
import pytest

import oracle
from oracle import moe as M
from tests import oracle_checks as C


def _ns(**override):
    d = dict(router_logits=M.router_logits, route=M.route, local_map=M.local_map, layout=M.layout,
             permute=M.permute, expert_ffn=M.expert_ffn, combine=M.combine)
    d.update(override)
    return types.SimpleNamespace(**d)


@pytest.mark.parametrize("check", C.ALL_CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check(_ns())


def test_layer_is_composition():
    rng = np.random.default_rng(11)
    T, E, k, H, I = 21, 10, 3, 8, 6
    x = rng.standard_normal((T, H)).astype(np.float32)
    logits = rng.standard_normal((T, E)).astype(np.float32)
    w_gu = rng.standard_normal((5, 2 * I, H)).astype(np.float32)
    w_dn = rng.standard_normal((5, H, I)).astype(np.float32)
    a = oracle.layer(logits, x, w_gu, w_dn, k, 2)
    b = C.compose_layer(_ns(), logits, x, w_gu, w_dn, k, 2)
    for key in b:
        assert np.array_equal(a[key], b[key]), key
    for t in range(T):
        out, idx, w = oracle.token_output(logits[t], x[t], w_gu, w_dn, k, 2)
        assert np.array_equal(idx, a["topk_idx"][t])
        assert np.allclose(out, a["out"][t], rtol=1e-12, atol=1e-12)


def test_empty_batch():
    res = oracle.layer(np.zeros((0, 8), np.float32), np.zeros((0, 4), np.float32), np.zeros((8, 6, 4), np.float32),
                       np.zeros((8, 4, 3), np.float32), 2, 0)
    assert res["out"].shape == (0, 4)
    assert res["counts"].sum() == 0 and res["offsets"][-1] == 0
    assert res["token_of_row"].size == 0


# ----------------------------------------------------------------------------- mutants


def _route_ties_high(logits, k):
    idx, w = M.route(logits[:, ::-1].copy(), k)
    E = logits.shape[1]
    return (E - 1 - idx).astype(np.int32), w


def _route_no_renorm(logits, k):
    idx, _ = M.route(logits, k)
    l = logits.astype(np.float64)
    p = np.exp(l - l.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    return idx, np.take_along_axis(p, idx.astype(np.int64), 1)


def _route_signed_zero(logits, k):
    # treats -0.0 as smaller than +0.0
    key = np.where((logits == 0) & np.signbit(logits), np.float32(-1e-30), logits)
    idx, _ = M.route(key, k)
    _, w = M.route(logits, k)
    return idx, w


def _route_ascending(logits, k):
    return M.route(-logits, k)


def _layout_desc(le, e_loc):
    counts, offsets, ros, tor = M.layout(le, e_loc)
    ros = ros.copy()
    for e in range(e_loc):
        a, b = offsets[e], offsets[e + 1]
        m = (ros >= a) & (ros < b)
        ros[m] = a + b - 1 - ros[m]
        tor[a:b] = tor[a:b][::-1]
    return counts, offsets, ros, tor


def _layout_inclusive(le, e_loc):
    counts, offsets, ros, tor = M.layout(le, e_loc)
    off2 = offsets.copy()
    off2[:-1] = offsets[1:]
    return counts, off2, ros, tor


def _layout_local_bug(le, e_loc):
    return M.layout(np.where(le >= 0, le, 0).astype(np.int32), e_loc)


def _ffn_silu_on_up(xp, offsets, w_gu, w_dn):
    I = w_gu.shape[1] // 2
    sw = np.concatenate([w_gu[:, I:], w_gu[:, :I]], axis=1)
    return M.expert_ffn(xp, offsets, sw, w_dn)


def _down(h, offsets, w_dn):
    y = np.zeros((h.shape[0], w_dn.shape[1]))
    for e in range(w_dn.shape[0]):
        a, b = offsets[e], offsets[e + 1]
        y[a:b] = h[a:b] @ w_dn[e].astype(np.float64).T
    return y


def _ffn_no_up_fixed(xp, offsets, w_gu, w_dn):
    I = w_gu.shape[1] // 2
    h = np.zeros((xp.shape[0], I))
    for e in range(w_gu.shape[0]):
        a, b = offsets[e], offsets[e + 1]
        g = xp[a:b].astype(np.float64) @ w_gu[e, :I].astype(np.float64).T
        h[a:b] = g / (1 + np.exp(-g))
    return h, _down(h, offsets, w_dn)


def _ffn_reshape_down(xp, offsets, w_gu, w_dn):
    E, H, I = w_dn.shape
    return M.expert_ffn(xp, offsets, w_gu, np.ascontiguousarray(w_dn).reshape(E, I, H).transpose(0, 2, 1))


def _ffn_sign(xp, offsets, w_gu, w_dn):
    I = w_gu.shape[1] // 2
    h = np.zeros((xp.shape[0], I))
    for e in range(w_gu.shape[0]):
        a, b = offsets[e], offsets[e + 1]
        x64 = xp[a:b].astype(np.float64)
        g = x64 @ w_gu[e, :I].astype(np.float64).T
        u = x64 @ w_gu[e, I:].astype(np.float64).T
        h[a:b] = g / (1 + np.exp(g)) * u
    return h, _down(h, offsets, w_dn)


def _permute_by_row(x, token_of_row):
    # gathers row r from x[r] instead of x[token_of_row[r]]
    R = len(token_of_row)
    return x[np.arange(R) % max(len(x), 1)] if len(x) else x[:0]


def _permute_next_token(x, token_of_row):
    return x[np.minimum(np.asarray(token_of_row, np.int64) + 1, len(x) - 1)]


def _combine_unweighted(y, w, ros, T, H):
    return M.combine(y, np.ones_like(w), ros, T, H)


def _combine_first_weight(y, w, ros, T, H):
    return M.combine(y, np.repeat(w[:, :1], w.shape[1], axis=1), ros, T, H)


def _combine_drop_last(y, w, ros, T, H):
    if ros.shape[1] <= 1:
        return M.combine(y, w * 0, ros, T, H)
    return M.combine(y, w[:, :-1], ros[:, :-1], T, H)


def _router_untransposed(x, w, bias=None):
    out = np.asarray(x, np.float64) @ np.asarray(w, np.float64).reshape(-1, np.asarray(w).shape[0])
    return out if bias is None else out + bias


def _router_no_bias(x, w, bias=None):
    return M.router_logits(x, w)


def _router_bias_subtracted(x, w, bias=None):
    return M.router_logits(x, w) - (0 if bias is None else np.asarray(bias, np.float64))


MUTANTS = {
    "router_weights_reshaped_not_transposed": dict(router_logits=_router_untransposed),
    "router_drops_bias": dict(router_logits=_router_no_bias),
    "router_bias_subtracted": dict(router_logits=_router_bias_subtracted),
    "route_ties_to_higher_id": dict(route=_route_ties_high),
    "route_no_renormalisation": dict(route=_route_no_renorm),
    "route_signed_zero_ordered": dict(route=_route_signed_zero),
    "route_smallest_logits": dict(route=_route_ascending),
    "layout_descending_tokens": dict(layout=_layout_desc),
    "layout_inclusive_offsets": dict(layout=_layout_inclusive),
    "layout_keeps_dropped_slots": dict(layout=_layout_local_bug),
    "ffn_silu_on_up": dict(expert_ffn=_ffn_silu_on_up),
    "ffn_missing_up_term": dict(expert_ffn=_ffn_no_up_fixed),
    "ffn_down_reshaped_not_transposed": dict(expert_ffn=_ffn_reshape_down),
    "ffn_silu_sign": dict(expert_ffn=_ffn_sign),
    "permute_gathers_by_row_index": dict(permute=_permute_by_row),
    "permute_next_token": dict(permute=_permute_next_token),
    "combine_unweighted": dict(combine=_combine_unweighted),
    "combine_first_weight_only": dict(combine=_combine_first_weight),
    "combine_drops_last_slot": dict(combine=_combine_drop_last),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    ns = _ns(**MUTANTS[name])
    failed = []
    for check in C.ALL_CHECKS:
        try:
            check(ns)
        except (AssertionError, ValueError, IndexError):
            failed.append(check.__name__)
    assert failed, f"planted mistake {name} passed every pin"
