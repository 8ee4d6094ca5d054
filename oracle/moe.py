"""Plain CPU oracle for one GPU's share of a phase-owned MoE expert layer.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product path (the
HIP library and its Python binding) never imports, calls or links it, and it
imports nothing from the product package.

What is computed, and where it comes from
-----------------------------------------
The paper (AInfer-PD, arXiv 2609.00993) runs its P and D batches through a
DeepEP-style expert layer: tokens are routed to their top-k experts
(Section 7.1 states top-8 routing over routed experts), dispatched to the
owners of those experts, run through the expert FFNs and combined back
(Section 2.2, "Parallel Organization of MoE Inference"; Section 5.2 splits
normal dispatch after expert notification, i.e. after the per-expert counts
are known and before routed data moves).  The paper does not write the
layer's arithmetic down, so this oracle uses the standard top-k softmax MoE
layer with SwiGLU experts, with every silent point fixed as follows:

* gate: softmax over the whole expert pool, then the k largest probabilities,
  renormalised over those k (renormalisation happens before dropping
  experts that live on other GPUs, so that summing every GPU's share gives
  the full layer, as expert parallelism requires);
* ties between equal logits go to the lower expert id; -0.0 equals +0.0;
  slot j of a token is its j-th largest logit;
* a GPU owns the expert block [e0, e0 + E_loc); slots routed elsewhere are
  dropped from this GPU's share;
* rows of one expert are laid out by ascending token index (a stable
  counting sort of the flattened slot index t*k + j), with no padding;
* expert e computes y = (silu(x W1^T) * (x W3^T)) W2^T, where W1 is rows
  [0, I) and W3 rows [I, 2I) of the gate/up matrix W_gu[e] of shape [2I, H]
  and W2 = W_dn[e] of shape [H, I]; silu(g) = g / (1 + exp(-g));
* the combined row is sum_j w[t, j] * y[row(t, j)] over the resident slots
  in slot order, or zero when no slot of t is resident.

All floating point is float64 (the inputs given as float32 / bfloat16 values
are upcast exactly).  Integer work (indices, counts, layout) is exact.
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "router_logits",
    "route",
    "local_map",
    "layout",
    "permute",
    "expert_ffn",
    "combine",
    "layer",
    "token_output",
]


def router_logits(x: np.ndarray, w_router: np.ndarray, bias=None) -> np.ndarray:
    """The gate's logits from hidden states: logits[t, e] = sum_h x[t, h]
    w_router[e, h] (+ bias[e]), in float64.  x: [T, H]; w_router: [E, H] (row
    e = expert e's gate vector); bias: [E] or None.  The paper routes tokens
    to their top-k experts (Section 7.1); the gate reads the token's hidden
    state through one linear map."""
    x64 = np.asarray(x, np.float64)
    w64 = np.asarray(w_router, np.float64)
    out = x64 @ w64.T
    if bias is not None:
        out = out + np.asarray(bias, np.float64)[None, :]
    return out


def route(logits: np.ndarray, k: int):
    """Top-k gating with renormalised softmax weights.

    logits: [T, E] float32 (finite).  Returns (topk_idx [T, k] int32 global
    expert ids, topk_w [T, k] float64).

    Step 1 (selection): order the experts of each token by the key
    (-logit, expert id) and keep the first k.  A stable sort on -logit keeps
    equal logits in ascending id order, and -0.0 compares equal to +0.0.
    Step 2 (weights): p = softmax over all E experts (max-subtracted), then
    w_j = p[idx_j] / sum_{i<k} p[idx_i].
    """
    logits = np.asarray(logits)
    T, E = logits.shape
    if not (1 <= k <= E):
        raise ValueError("top-k needs 1 <= k <= E")
    if T == 0:
        return np.zeros((0, k), np.int32), np.zeros((0, k), np.float64)
    order = np.argsort(-logits, axis=1, kind="stable")
    topk_idx = order[:, :k].astype(np.int32)

    l64 = logits.astype(np.float64)
    m = l64.max(axis=1, keepdims=True)
    p = np.exp(l64 - m)
    p = p / p.sum(axis=1, keepdims=True)
    sel = np.take_along_axis(p, topk_idx.astype(np.int64), axis=1)
    topk_w = sel / sel.sum(axis=1, keepdims=True)
    return topk_idx, topk_w


def local_map(topk_idx: np.ndarray, e0: int, e_loc: int) -> np.ndarray:
    """Global expert id -> local id on the GPU owning [e0, e0+E_loc), else -1."""
    le = topk_idx.astype(np.int64) - e0
    return np.where((le >= 0) & (le < e_loc), le, -1).astype(np.int32)


def layout(le: np.ndarray, e_loc: int):
    """Dispatch layout: per-expert histogram, prefix sum, stable row ranks.

    le: [T, k] local expert ids (-1 = not on this GPU).  Returns
    counts [E_loc], offsets [E_loc+1], row_of_slot [T, k] (-1 = dropped) and
    token_of_row [R] where R = offsets[E_loc].

    This is the notification half of normal dispatch (Section 5.2): once the
    counts and offsets are known the shape of the dispatch is fixed.  The row
    of slot (t, j) routed to local expert e is
        offsets[e] + #{ slots (t', j') before (t, j) in t*k+j order with expert e }
    which, since a token picks an expert at most once, is the number of
    earlier tokens routed to e.
    """
    T, k = le.shape
    flat = le.reshape(-1).astype(np.int64)
    S = flat.size
    # histogram
    counts = np.zeros(e_loc, np.int64)
    for e in range(e_loc):
        counts[e] = int(np.count_nonzero(flat == e))
    # exclusive prefix sum
    offsets = np.zeros(e_loc + 1, np.int64)
    for e in range(e_loc):
        offsets[e + 1] = offsets[e] + counts[e]
    # rank of each slot among the earlier slots of the same expert
    row_of_slot = np.full(S, -1, np.int64)
    for e in range(e_loc):
        hit = flat == e
        before = np.cumsum(hit) - hit  # number of earlier slots with expert e
        row_of_slot[hit] = offsets[e] + before[hit]
    R = int(offsets[e_loc])
    token_of_row = np.full(R, -1, np.int64)
    kept = row_of_slot >= 0
    token_of_row[row_of_slot[kept]] = np.nonzero(kept)[0] // k
    return (
        counts.astype(np.int32),
        offsets.astype(np.int32),
        row_of_slot.reshape(T, k).astype(np.int32),
        token_of_row.astype(np.int32),
    )


def permute(x: np.ndarray, token_of_row: np.ndarray) -> np.ndarray:
    """Data-movement half of dispatch: x_perm[row] = x[token_of_row[row]]."""
    return x[token_of_row.astype(np.int64)]


def _silu(g: np.ndarray) -> np.ndarray:
    return g / (1.0 + np.exp(-g))


def expert_ffn(x_perm: np.ndarray, offsets: np.ndarray, w_gu: np.ndarray, w_dn: np.ndarray):
    """Grouped SwiGLU expert FFN over expert-contiguous rows, in float64.

    x_perm [R, H]; w_gu [E_loc, 2I, H] (rows [0, I) gate W1, [I, 2I) up W3);
    w_dn [E_loc, H, I].  Returns (h [R, I], y [R, H]) with
    h = silu(x W1^T) * (x W3^T) and y = h W2^T, rows of expert e being
    [offsets[e], offsets[e+1]).
    """
    x_perm = np.asarray(x_perm, np.float64)
    e_loc, two_i, H = w_gu.shape
    I = two_i // 2
    R = x_perm.shape[0]
    h = np.zeros((R, I), np.float64)
    y = np.zeros((R, H), np.float64)
    for e in range(e_loc):
        a, b = int(offsets[e]), int(offsets[e + 1])
        if a == b:
            continue
        xe = x_perm[a:b]
        w1 = np.asarray(w_gu[e, :I], np.float64)
        w3 = np.asarray(w_gu[e, I:], np.float64)
        w2 = np.asarray(w_dn[e], np.float64)
        g = xe @ w1.T
        u = xe @ w3.T
        h[a:b] = _silu(g) * u
        y[a:b] = h[a:b] @ w2.T
    return h, y


def combine(y: np.ndarray, topk_w: np.ndarray, row_of_slot: np.ndarray, T: int, H: int) -> np.ndarray:
    """Weighted combine: out[t] = sum_j w[t, j] y[row(t, j)] over resident slots,
    accumulated in slot order; rows with no resident slot are zero."""
    out = np.zeros((T, H), np.float64)
    k = row_of_slot.shape[1] if row_of_slot.ndim == 2 else 0
    for j in range(k):
        r = row_of_slot[:, j].astype(np.int64)
        kept = r >= 0
        out[kept] += topk_w[kept, j][:, None] * np.asarray(y[r[kept]], np.float64)
    return out


def layer(logits, x, w_gu, w_dn, k: int, e0: int):
    """The whole layer for one phase batch; returns a dict of every stage."""
    x = np.asarray(x)
    T, H = x.shape
    e_loc = w_gu.shape[0]
    topk_idx, topk_w = route(logits, k)
    le = local_map(topk_idx, e0, e_loc)
    counts, offsets, row_of_slot, token_of_row = layout(le, e_loc)
    x_perm = permute(x, token_of_row)
    h, y = expert_ffn(x_perm, offsets, w_gu, w_dn)
    out = combine(y, topk_w, row_of_slot, T, H)
    return dict(
        topk_idx=topk_idx,
        topk_w=topk_w,
        local=le,
        counts=counts,
        offsets=offsets,
        row_of_slot=row_of_slot,
        token_of_row=token_of_row,
        x_perm=x_perm,
        h=h,
        y=y,
        out=out,
    )


def token_output(logits_row, x_row, w_gu, w_dn, k: int, e0: int):
    """The layer output of a single token, from its own logits and hidden row.

    Used to check sampled tokens of batches too large for the full oracle;
    the output of a token does not depend on the other tokens of its batch.
    Returns (out_row [H] float64, topk_idx [k], topk_w [k]).
    """
    idx, w = route(np.asarray(logits_row)[None, :], k)
    idx, w = idx[0], w[0]
    e_loc, two_i, H = w_gu.shape
    I = two_i // 2
    xr = np.asarray(x_row, np.float64)
    out = np.zeros(H, np.float64)
    for j in range(k):
        le = int(idx[j]) - e0
        if not (0 <= le < e_loc):
            continue
        g = np.asarray(w_gu[le, :I], np.float64) @ xr
        u = np.asarray(w_gu[le, I:], np.float64) @ xr
        hh = _silu(g) * u
        out += w[j] * (np.asarray(w_dn[le], np.float64) @ hh)
    return out, idx, w
