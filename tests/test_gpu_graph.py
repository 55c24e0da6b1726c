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
