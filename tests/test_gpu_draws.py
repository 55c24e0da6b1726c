"""RandomNode and UniformChoice of Algorithm 1 (Section 3.3) as the library
draws them on the GPU: uniform over the candidates, at 10^5 and more draws
per candidate set. The GPU's draws equal the oracle's bit for bit (the
parity tests); these check the distribution of the library's own outputs at
full size, where the oracle would be slow."""
import numpy as np
import pytest
import torch
from scipy.stats import chisquare

from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import pipeline as PL
from paper_2609_36959_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    B.lib()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def test_node_and_rank_draws_at_2_20_tokens():
    """Three nodes of three ranks. Every token comes from node 0, which holds
    none of its experts: e0 lives on node 1 only (ranks 3, 4, 5), e1 on node
    2 only (rank 6), e2 on nodes 1 and 2 (ranks 3 and 7, 8). The cover is
    {1, 2}; e2 draws node 1 or 2 with equal odds, then a rank of that node
    holding it; e0 draws one of three ranks."""
    N, g, E = 3, 3, 3
    table = np.full((9, 2), -1, np.int32)
    table[3] = [0, 2]
    table[4, 0] = 0
    table[5, 0] = 0
    table[6, 0] = 1
    table[7, 0] = 2
    table[8, 0] = 2
    L = B.cobalt_layout_create(N, g, E, 2, table)
    T = 1 << 20
    print(f"draws T={T}", flush=True)
    topk = torch.tensor([[0, 1, 2]], dtype=torch.int32, device="cuda").repeat(T, 1).contiguous()
    src = torch.zeros(T, dtype=torch.int32, device="cuda")
    a = torch.empty(T, 3, dtype=torch.int32, device="cuda")
    rn = torch.empty(T, dtype=torch.int16, device="cuda")
    B.cobalt_assign(L, topk, src, 2024, 7, 0, a, rn)
    torch.cuda.synchronize()
    assert bool((rn == 0b110).all().item())
    c0 = torch.bincount(a[:, 0].long(), minlength=9).cpu().numpy()
    assert c0[[0, 1, 2, 6, 7, 8]].sum() == 0
    assert chisquare(c0[3:6]).pvalue > 1e-4            # e0: ranks 3, 4, 5
    assert bool((a[:, 1] == 6).all().item())            # e1: its only holder
    c2 = torch.bincount(a[:, 2].long(), minlength=9).cpu().numpy()
    assert c2[[0, 1, 2, 4, 5, 6]].sum() == 0
    node1, node2 = c2[3], c2[7] + c2[8]
    assert chisquare([node1, node2]).pvalue > 1e-4      # RandomNode over the cover
    assert chisquare(c2[7:9]).pvalue > 1e-4             # UniformChoice on node 2
    assert min(c0[3:6].min(), node1, node2, c2[7:9].min()) >= 100000
    B.cobalt_layout_destroy(L)


def test_rank_draws_on_the_full_colocate_step():
    """colocate-e256 at full size (T = 131072): for every expert with two or
    more replicas on its node, the tasks it runs there are spread uniformly
    over those replicas (chi-square per expert with at least 10^5 tasks on
    a node, Bonferroni over the experts tested)."""
    w = W.WORKLOADS["colocate-e256"]
    print("draws colocate-e256 full size", flush=True)
    st = PL.RoutingStep(w, seed=w.seed, device="cuda")
    st.assign()
    torch.cuda.synchronize()
    e = st.topk.long().flatten()
    r = st.assigned.long().flatten()
    counts = torch.zeros(w.E * w.G, dtype=torch.int64, device="cuda")
    counts.index_add_(0, e * w.G + r, torch.ones_like(e))
    counts = counts.view(w.E, w.G).cpu().numpy()
    held = np.zeros((w.E, w.G), bool)
    for rank in range(w.G):
        held[[x for x in st.table[rank] if x >= 0], rank] = True
    tested = []
    for ex in range(w.E):
        for n in range(w.N):
            ranks = [n * w.g + i for i in range(w.g) if held[ex, n * w.g + i]]
            c = counts[ex, ranks]
            assert counts[ex, n * w.g:(n + 1) * w.g].sum() == c.sum()  # only holders
            if len(ranks) >= 2 and c.sum() >= 100000:
                tested.append(chisquare(c).pvalue)
    assert tested, "no expert with enough replicated tasks"
    assert min(tested) > 1e-4 / len(tested)
    st.close()
