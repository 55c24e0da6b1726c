"""Pins of the oracle's per-replica workload (Section 3.1, w_er) and of the
Stage-2 intra-node rebalancing (Section 3.2: greedy bin-packing of a node's
replicas, heaviest first, onto the least-loaded eligible rank)."""
import itertools

import numpy as np
import pytest

import oracle
from paper_2609_36959_amd import workload as W


def test_replica_load_is_a_pair_histogram():
    rng = np.random.default_rng(3)
    T, K, E, G = 500, 4, 12, 6
    topk = rng.integers(0, E, size=(T, K)).astype(np.int32)
    a = rng.integers(0, G, size=(T, K)).astype(np.int32)
    a[0, 0] = -1  # skipped
    want = np.zeros((E, G), np.int64)
    ok = a >= 0
    np.add.at(want, (topk[ok], a[ok]), 1)
    got = oracle.replica_load(topk, a, E, G)
    assert np.array_equal(got.astype(np.int64), want)
    got = oracle.replica_load(topk, a, E, G, got)  # accumulates
    assert np.array_equal(got.astype(np.int64), 2 * want)


def test_replica_load_sums_match_rank_loads():
    w = W.with_sizes(W.WORKLOADS["clusters-e64"], T=32 * 64)
    table, owner = W.layout(w, w.seed)
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    topk = W.routing(w, w.seed)[0].numpy()
    a, _ = oracle.assign(w.N, w.g, w.E, tabs, topk, seed=1)
    load = oracle.replica_load(topk, a, w.E, w.G).astype(np.int64)
    _, _, rank_load = oracle.traffic(a, w.N, w.g)
    assert np.array_equal(load.sum(0), rank_load)
    assert load.sum() == w.T * w.K
    held = np.zeros((w.E, w.G), bool)
    for r in range(w.G):
        held[table[r][table[r] >= 0], r] = True
    assert np.all(load[~held] == 0)  # tasks only land on replicas (Eq. 2)


def _one_node_table(experts_per_rank, S):
    g = len(experts_per_rank)
    t = np.full((g, S), -1, np.int32)
    for r, es in enumerate(experts_per_rank):
        t[r, : len(es)] = es
    return t


def test_lpt_textbook_example():
    """Two ranks, five distinct replicas of loads 5,4,3,3,3: the greedy
    gives 10 (optimum 9, within the 7/6 bound for two machines)."""
    E, S = 5, 5
    table = _one_node_table([[0, 1, 2], [3, 4]], S)
    load = np.zeros((E, 2), np.float32)
    load[0, 0], load[1, 0], load[2, 0], load[3, 1], load[4, 1] = 5, 4, 3, 3, 3
    new, own, rl = oracle.intra_node_rebalance(1, 2, E, table, None, load)
    assert sorted(rl.tolist()) == [8.0, 10.0]
    assert sorted(new[0][new[0] >= 0].tolist()) == [0, 3]  # 5 then 3
    assert sorted(new[1][new[1] >= 0].tolist()) == [1, 2, 4]


def _brute_opt(loads, g):
    best = None
    for assign in itertools.product(range(g), repeat=len(loads)):
        m = max(sum(l for l, a in zip(loads, assign) if a == i) for i in range(g))
        best = m if best is None else min(best, m)
    return best


@pytest.mark.parametrize("case", range(25))
def test_within_lpt_bound_of_brute_force_optimum(case):
    """Distinct experts and ample slots make Stage 2 plain longest-processing-
    time scheduling, so its makespan is at most (4/3 - 1/(3g)) of optimal."""
    rng = np.random.default_rng(case)
    g = int(rng.integers(2, 4))
    n = int(rng.integers(2, 8))
    E = n
    per = [list(range(i, n, g)) for i in range(g)]
    table = _one_node_table(per, n)
    load = np.zeros((E, g), np.float32)
    loads = rng.integers(1, 20, size=n).astype(np.float32)
    for r in range(g):
        for e in per[r]:
            load[e, r] = loads[e]
    _, _, rl = oracle.intra_node_rebalance(1, g, E, table, None, load)
    opt = _brute_opt(loads.tolist(), g)
    assert rl.max() <= (4 / 3 - 1 / (3 * g)) * opt + 1e-6
    assert abs(rl.sum() - loads.sum()) < 1e-3


def test_validity_conservation_and_owners_on_workloads():
    for name in ("tiny", "clusters-e64", "colocate-e256", "drift-e384"):
        w = W.WORKLOADS[name]
        table, owner = W.layout(w, w.seed)
        rng = np.random.default_rng(7)
        load = rng.gamma(1.0, 100.0, size=(w.E, w.G)).astype(np.float32)
        new, own, rl = oracle.intra_node_rebalance(w.N, w.g, w.E, table, owner, load)
        nm, rm, _ = oracle.layout_tables(w.N, w.g, w.E, new, own)  # valid, owners hold
        _, rm0, _ = oracle.layout_tables(w.N, w.g, w.E, table, owner)
        pc = np.vectorize(lambda v: bin(int(v)).count("1"))
        assert np.array_equal(pc(rm), pc(rm0))  # replicas per (expert, node) unchanged
        assert np.all((new >= 0).sum(1) <= w.S)


def test_stuck_node_keeps_its_placement():
    """Rank 0 holds {a, b}, rank 1 holds {a, c} (S = 2). Heaviest first:
    a(9) -> rank 0, b(8) -> rank 1, c(7) -> rank 1 (now full); the second a
    finds rank 0 holding a and rank 1 full, so the node keeps its layout."""
    a, b, c = 0, 1, 2
    table = _one_node_table([[a, b], [a, c]], 2)
    load = np.zeros((3, 2), np.float32)
    load[a, 0], load[b, 0], load[c, 1], load[a, 1] = 9, 8, 7, 1
    new, own, rl = oracle.intra_node_rebalance(1, 2, 3, table, None, load)
    assert np.array_equal(new, table)
    assert rl.tolist() == [17.0, 8.0]
    # with a lighter b the greedy completes and moves replicas
    load[b, 0] = 0.5
    new, own, rl = oracle.intra_node_rebalance(1, 2, 3, table, None, load)
    assert sorted(rl.tolist()) == [8.0, 9.5]
    assert own[a] in (0, 1) and a in new[own[a]]


def test_rejects_bad_loads():
    table = _one_node_table([[0], [1]], 1)
    load = np.full((2, 2), np.nan, np.float32)
    load[0, 0] = 1
    with pytest.raises(oracle.OracleError):
        oracle.intra_node_rebalance(1, 2, 2, table, None, load)
    load[1, 1] = -1
    with pytest.raises(oracle.OracleError):
        oracle.intra_node_rebalance(1, 2, 2, table, None, load)
