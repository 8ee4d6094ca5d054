"""The allocation-free dispatch layout (moe_dispatch_layout_noalloc) against
the context's moe_dispatch_layout, through the C ABI, on calls in a row that
share the device's scratch array: a batch of many histogram chunks, a smaller
batch of fewer chunks, a one-chunk batch, and an empty one.  Results are
integers and must be equal; both are also checked against the oracle's
layout of the same routing."""

import numpy as np
import pytest

import oracle
from synth import BF16, LayerSpec, make_layer
from tests.gpu_util import GpuLayer, read_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_noalloc_layout_matches_context_layout():
    import torch

    from paper_2609_00993_amd import moepd as M

    spec = LayerSpec("noalloc", E=64, e0=16, E_loc=32, k=8, H=64, I=64, dtype=BF16, T_P=3000, T_D=100)
    inp = make_layer(spec, seed=31)
    g = GpuLayer(inp)
    k, e0, E_loc = spec.k, spec.e0, spec.E_loc
    cap = spec.T_P * min(k, E_loc)
    dev = torch.device("cuda")
    counts = torch.empty(E_loc, dtype=torch.int32, device=dev)
    offsets = torch.empty(E_loc + 1, dtype=torch.int32, device=dev)
    ros = torch.empty(spec.T_P * k, dtype=torch.int32, device=dev)
    tor = torch.empty(cap, dtype=torch.int32, device=dev)
    s = torch.cuda.Stream()
    try:
        # (phase, tokens): 3000 tokens = 24000 slots in many chunks, then 1000
        # (fewer chunks), then 100 on the D phase (one chunk), then none
        for ph, T in ((0, 3000), (0, 1000), (1, 100), (1, 0)):
            print(f"[noalloc] phase {ph} T={T}", flush=True)
            lg = g.logits[ph][:T] if T else None
            M.check(M.moe_route(g.ctx, ph, lg, T, g.streams[ph]))
            M.check(M.moe_dispatch_layout(g.ctx, ph, g.streams[ph]))
            torch.cuda.synchronize()
            st, v = M.moe_phase_view(g.ctx, ph)
            M.check(st)
            ref_counts = read_dev(v.counts, (E_loc,), np.int32)
            ref_offsets = read_dev(v.offsets, (E_loc + 1,), np.int32)
            R = int(ref_offsets[-1])
            ref_ros = read_dev(v.row_of_slot, (T, k), np.int32)
            ref_tor = read_dev(v.token_of_row, (R,), np.int32)
            for t in (counts, offsets, ros, tor):
                t.fill_(-7)
            torch.cuda.synchronize()
            M.check(M.moe_dispatch_layout_noalloc(v.topk_idx if T else None, T, k, e0, E_loc, counts, offsets,
                                                  ros if T else None, tor if T else None, s),
                    "moe_dispatch_layout_noalloc")
            torch.cuda.synchronize()
            got_counts, got_offsets = counts.cpu().numpy(), offsets.cpu().numpy()
            got_ros = ros.cpu().numpy()[:T * k].reshape(T, k)
            got_tor_all = tor.cpu().numpy()
            assert np.array_equal(got_counts, ref_counts), (T, "counts")
            assert np.array_equal(got_offsets, ref_offsets), (T, "offsets")
            assert np.array_equal(got_ros, ref_ros), (T, "row_of_slot")
            assert np.array_equal(got_tor_all[:R], ref_tor), (T, "token_of_row")
            assert np.all(got_tor_all[R:] == -7), (T, "token_of_row written past R")
            # both against the oracle's layout of the same routing
            idx, _ = oracle.route(inp.logits[ph][:T], k)
            o_counts, o_offsets, o_ros, o_tor = oracle.layout(oracle.local_map(idx, e0, E_loc), E_loc)
            assert np.array_equal(got_counts, o_counts) and np.array_equal(got_offsets, o_offsets)
            assert np.array_equal(got_ros, o_ros) and np.array_equal(got_tor_all[:R], o_tor)
            M.check(M.moe_phase_reset(g.ctx, ph))
    finally:
        g.close()


def test_noalloc_refuses_bad_arguments():
    import torch

    from paper_2609_00993_amd import moepd as M

    s = torch.cuda.Stream()
    buf = torch.zeros(64, dtype=torch.int32, device="cuda")
    ok = dict(topk_idx=buf, T=4, top_k=2, expert_begin=0, num_local_experts=8, counts=buf, offsets=buf,
              row_of_slot=buf, token_of_row=buf, stream=s)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return M.moe_dispatch_layout_noalloc(**a)

    assert call(T=-1) == M.MOE_ERR_INVALID_ARG
    assert call(top_k=0) == M.MOE_ERR_INVALID_ARG
    assert call(top_k=17) == M.MOE_ERR_INVALID_ARG
    assert call(num_local_experts=257) == M.MOE_ERR_INVALID_ARG
    assert call(counts=None) == M.MOE_ERR_INVALID_ARG
    assert call(stream=None) == M.MOE_ERR_INVALID_ARG
    assert call(topk_idx=None) == M.MOE_ERR_INVALID_ARG
    assert call(T=(1 << 20) + 1) == M.MOE_ERR_CAPACITY
