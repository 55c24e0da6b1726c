"""GPU parity of Algorithm 1 (Section 3.3) on layouts where experts sit on
many nodes, so that the minimum-cover search runs deep: remote covers of
three and more nodes, ties between several minimum covers, experts held on
every node but one (the whole remote mask), and E not a multiple of G. Node
counts 10, 12 and 16 take the kernel's 16-bit SWAR lanes, N <= 9 its 8-bit
lanes; K is 8 or 16. Both assignment modes, and the rest of the path, are
compared bit for bit with the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import workload as W
from test_gpu_parity import check_against_oracle

SPREADS = ("dense", "sparse", "mixed", "allbutone")


def dense_layout(N, g, E, spread, seed):
    """Owner of expert e is rank e % G; each expert then gets replicas on a
    seeded number of further nodes, on a random rank of each. Returns
    (slot_table [G][S], owner [E]) with S the fullest rank's count."""
    rng = np.random.default_rng(seed)
    G = N * g
    slots = [[] for _ in range(G)]
    owner = (np.arange(E) % G).astype(np.int32)
    for e in range(E):
        slots[owner[e]].append(e)
        home = owner[e] // g
        if spread == "dense":
            h = int(rng.integers(3, N + 1))
        elif spread == "sparse":
            h = int(rng.choice([1, 2, 3]))
        elif spread == "mixed":
            h = int(rng.choice([1, 1, 2, 3, max(1, N // 2), N - 1, N]))
        else:  # allbutone: on every node except one, chosen at random
            h = N - 1
        others = [n for n in range(N) if n != home]
        if spread == "allbutone":
            missing = int(rng.integers(N))
            nodes = [n for n in range(N) if n != missing]
            if home == missing:  # the owner's node holds it: drop another instead
                nodes = [n for n in range(N) if n != others[int(rng.integers(len(others)))]]
        else:
            nodes = [home] + list(rng.choice(others, size=min(h, N) - 1, replace=False))
        for n in nodes:
            if n == home:
                continue
            r = n * g + int(rng.integers(g))
            slots[r].append(e)
    S = max(len(s) for s in slots)
    table = np.full((G, S), -1, np.int32)
    for r in range(G):
        table[r, : len(slots[r])] = slots[r]
    return table, owner


def routing(E, K, T, seed):
    rng = np.random.default_rng(seed)
    topk = np.argsort(rng.random((T, E)), axis=1)[:, :K].astype(np.int32)
    g_ = rng.random((T, K)).astype(np.float32) + 0.05
    return topk, (g_ / g_.sum(1, keepdims=True)).astype(np.float32)


CASES = [
    # N, g, E, K, tokens per rank, source ranks, spread
    (10, 2, 37, 8, 40, "ragged", "sparse"),
    (10, 1, 45, 16, 90, "null", "mixed"),
    (12, 2, 50, 8, 40, "null", "dense"),
    (12, 1, 29, 16, 80, "ragged", "sparse"),
    (16, 2, 100, 8, 30, "null", "allbutone"),
    (16, 1, 40, 16, 60, "ragged", "sparse"),
    (16, 4, 203, 16, 20, "null", "mixed"),
    (16, 1, 16, 16, 50, "null", "sparse"),   # K = E: every token selects every expert
    (16, 2, 77, 8, 40, "ragged", "dense"),
    (9, 2, 31, 8, 50, "ragged", "sparse"),
    (5, 3, 17, 16, 60, "null", "mixed"),
    (8, 8, 70, 8, 20, "null", "allbutone"),
]


def case_inputs(N, g, E, K, per_rank, srckind, spread):
    seed = N * 1000 + E * 10 + K
    G = N * g
    T = G * per_rank + (7 if srckind == "ragged" else 0)
    table, owner = dense_layout(N, g, E, spread, seed)
    topk, gates = routing(E, K, T, seed + 1)
    src = None if srckind == "null" else W.ragged_src(T, G, seed=seed)
    w = W.Workload("dense-cover", T, E, K, 64, N, g, table.shape[1])
    return w, seed, topk, gates, table, owner, src


def test_cases_reach_deep_covers():
    """On the CPU: the cases above do exercise what they are meant to (remote
    covers of three or more nodes, whole remote masks, E not a multiple of
    G), as the oracle computes them."""
    deepest, whole_mask, ragged_e = 0, False, False
    for N, g, E, K, per_rank, srckind, spread in CASES:
        w, seed, topk, gates, table, owner, src = case_inputs(N, g, E, K, per_rank, srckind,
                                                               spread)
        tabs = oracle.layout_tables(N, g, E, table, owner)
        _, rn = oracle.assign(N, g, E, tabs, topk, src, seed=seed, step=0)
        pc = np.array([bin(int(v)).count("1") for v in rn])
        deepest = max(deepest, int(pc.max()))
        ragged_e |= E % (N * g) != 0
        node_mask = tabs[0]
        whole_mask |= any(bin(int(m)).count("1") == N - 1 for m in node_mask)
        if N >= 10 and spread in ("sparse", "mixed"):
            assert (pc >= 3).mean() > 0.2, (N, E, K, spread)
    assert deepest >= 6 and whole_mask and ragged_e


@pytest.mark.gpu
@pytest.mark.parametrize("N,g,E,K,per_rank,srckind,spread", CASES)
def test_dense_cover_parity(N, g, E, K, per_rank, srckind, spread):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    B.lib()
    w, seed, topk, gates, table, owner, src = case_inputs(N, g, E, K, per_rank, srckind, spread)
    print(f"dense cover N={N} g={g} E={E} K={K} T={w.T} src={srckind} spread={spread}",
          flush=True)
    for step in (0, 5):
        check_against_oracle(w, seed, topk, gates, table, owner, src, step=step, mode=0)
    check_against_oracle(w, seed, topk, gates, table, owner, src, step=0, mode=1)
