"""D-phase graph capture and replay (GPU, through the C ABI).

The paper's D path replays captured graphs against the phase's stable
buffers (Section 6.1).  A D layer captured once and replayed must give the
eager layer's bits on every replay, with the other phase's eager work and
host synchronisations between replays.
"""
import numpy as np
import pytest

from synth import make_config
from tests.gpu_util import GpuLayer
from tests.test_gpu_layer import check_phase

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _d_state(g):
    res = g.fetch(1)
    return {k: res[k].copy() for k in ("topk_idx", "topk_w", "counts", "offsets", "row_of_slot", "token_of_row",
                                       "x_perm_raw", "h_raw", "y", "out")}


@pytest.mark.parametrize("d_priority_us", [0, 300])
def test_d_layer_graph_replays_match_eager(d_priority_us):
    import torch

    inp = make_config(1)
    g = GpuLayer(inp, d_priority_us=d_priority_us)
    try:
        M = g.M
        sg = torch.cuda.Stream()
        # eager D on the capture stream first (the phase last ran there)
        g.run(1, stream=sg)
        torch.cuda.synchronize()
        ref = _d_state(g)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=sg):
            M.layer(g.ctx, 1, g.logits[1], g.T[1], g.x[1], g.out[1], sg)
        torch.cuda.synchronize()
        for rep in range(3):
            g.out[1].zero_()
            g.run(0)  # the P phase, eager, on its own stream
            torch.cuda.synchronize()
            with torch.cuda.stream(sg):
                graph.replay()
            torch.cuda.synchronize()
            got = _d_state(g)
            for key in ref:
                assert np.array_equal(got[key], ref[key]), (rep, key)
        # replay concurrently with eager P, then check once more
        g.out[1].zero_()
        torch.cuda.synchronize()
        g.run(0)
        with torch.cuda.stream(sg):
            graph.replay()
        torch.cuda.synchronize()
        got = _d_state(g)
        for key in ref:
            assert np.array_equal(got[key], ref[key]), ("concurrent", key)
        # the replayed D layer (every stage) and the eager P layer beside it
        # against the oracle
        check_phase(g, inp, 1)
        check_phase(g, inp, 0)
        # the eager API still works on the phase after the replays
        g.run(1, stream=sg)
        torch.cuda.synchronize()
        assert np.array_equal(_d_state(g)["out"], ref["out"])
        del graph
    finally:
        g.close()


@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")
def test_capture_refuses_a_stream_hand_over():
    """A phase last driven on one stream cannot start a capture on another:
    the hand-over wait could not be part of the graph."""
    import torch

    inp = make_config(1)
    g = GpuLayer(inp)
    try:
        M = g.M
        g.run(1)  # the phase's stream is now g.streams[1]
        torch.cuda.synchronize()
        sg = torch.cuda.Stream()
        graph = torch.cuda.CUDAGraph()
        st = None
        with torch.cuda.graph(graph, stream=sg):
            st = M.moe_route(g.ctx, 1, g.logits[1], g.T[1], sg)
        assert st == M.MOE_ERR_STATE
        torch.cuda.synchronize()
        # nothing was enqueued and the phase is still usable from its stream
        g.run(1)
        torch.cuda.synchronize()
        del graph
    finally:
        g.close()
