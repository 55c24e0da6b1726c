"""The four calls of a step captured in a HIP graph: every replay, with new
inputs written eagerly between replays, must equal an eager run on the same
inputs (the kernels clear their own scratch; nothing records a memset)."""
import numpy as np
import pytest
import torch

from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import pipeline as PL
from paper_2609_36959_amd import workload as W

pytestmark = pytest.mark.gpu


def snapshot(st):
    return [t.clone() for t in (st.coact, st.count, st.assigned, st.remote, st.counts,
                                st.offsets, st.pos, st.packed, st.y)]


@pytest.mark.parametrize("name,T", [("tiny", 4096), ("colocate-e128", 32 * 96)])
def test_graph_replays_match_eager(name, T):
    assert torch.cuda.is_available()
    B.lib()
    w = W.with_sizes(W.WORKLOADS[name], T=T)
    st = PL.RoutingStep(w, seed=w.seed, device="cuda", route_device="cpu")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        st.run()
    torch.cuda.synchronize()
    for rep in range(3):
        # new inputs, written eagerly into the captured buffers
        topk, gates = W.routing(w, w.seed, step=rep + 1)
        st.topk.copy_(topk)
        st.gates.copy_(gates)
        st.x.copy_(W.hidden(w, w.seed, step=rep + 1))
        st.coact.zero_()
        st.count.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = snapshot(st)
        st.coact.zero_()
        st.count.zero_()
        st.run()
        torch.cuda.synchronize()
        for a, b in zip(got, snapshot(st)):
            assert torch.equal(a, b), f"replay {rep} differs from the eager run"
    del g
    st.close()


def extended(st):
    """The step and every call outside it, in one sequence."""
    st.run()
    st.node_pack()
    st.node_combine()
    st.load()
    st.ema(0.9, B.EMA_CLEAR)


def bits(t):
    return t.view({2: torch.int16, 4: torch.int32, 8: torch.int64}[t.element_size()]) \
        if t.is_floating_point() else t


def snapshot_all(st):
    return snapshot(st) + [t.clone() for t in (
        st.node_counts, st.node_offsets, st.node_pos, st.node_packed, st.node_partial, st.y_node,
        st.replica_load, st.ema_coact, st.ema_count, st.ochiai)]


@pytest.mark.parametrize("name,T", [("tiny", 4096), ("colocate-e128", 32 * 96)])
def test_graph_of_every_call_matches_eager(name, T):
    """Node-deduplicated pack, node-level combine, replica loads and the EMA
    update with clearing, captured with the step: every replay equals the
    eager sequence on the same inputs and the same starting state."""
    assert torch.cuda.is_available()
    B.lib()
    w = W.with_sizes(W.WORKLOADS[name], T=T)
    st = PL.RoutingStep(w, seed=w.seed, device="cuda", route_device="cpu")
    extended(st)  # allocates the lazily created buffers before the capture
    torch.cuda.synchronize()
    ema0 = (st.ema_coact.clone() + 3.0, st.ema_count.clone() + 5.0)

    def reset():
        st.coact.zero_()
        st.count.zero_()
        st.replica_load.zero_()
        st.ema_coact.copy_(ema0[0])
        st.ema_count.copy_(ema0[1])

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        extended(st)
    torch.cuda.synchronize()
    for rep in range(3):
        topk, gates = W.routing(w, w.seed, step=rep + 1)
        st.topk.copy_(topk)
        st.gates.copy_(gates)
        st.x.copy_(W.hidden(w, w.seed, step=rep + 1))
        reset()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = snapshot_all(st)
        reset()
        extended(st)
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(got, snapshot_all(st))):
            # bit patterns: rows past the used ones hold whatever the buffer
            # held before, NaN patterns included, in both runs alike
            assert torch.equal(bits(a), bits(b)), f"replay {rep}: output {i} differs from the eager run"
    del g
    st.close()
