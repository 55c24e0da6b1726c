"""Pins of the oracle's layout tables and communication-aware task
assignment (Section 3.3, Algorithm 1; Eq. 1 and Eq. 2 of Section 3.1)."""
import itertools

import numpy as np
import pytest
from scipy.stats import chisquare

import oracle
from paper_2609_36959_amd import workload as W


def popcount(v):
    return bin(int(v)).count("1")


# ------------------------------------------------------------------ Fig. 1
def test_fig1_layout_tables(fig1):
    nm, rm, own = oracle.layout_tables(fig1["N"], fig1["g"], fig1["E"], fig1["table"])
    reps = [sum(popcount(rm[e, n]) for n in range(fig1["N"])) for e in range(fig1["E"])]
    assert reps == fig1["replicas"]  # caption: 3, 2, 2, 1 replicas
    assert own.tolist() == [0, 0, 1, 3]  # lowest rank holding each expert
    _, _, own2 = oracle.layout_tables(fig1["N"], fig1["g"], fig1["E"], fig1["table"], fig1["owner"])
    assert own2.tolist() == fig1["owner"].tolist()


@pytest.mark.parametrize("seed", [0, 1, 2, 99])
def test_fig1_hand_cases(fig1, seed):
    N, g, E = fig1["N"], fig1["g"], fig1["E"]
    tabs = oracle.layout_tables(N, g, E, fig1["table"], fig1["owner"])
    rows = np.array(fig1["tokens"], np.int64)
    src = rows[:, 1].astype(np.int32)
    topk = rows[:, 2:4].astype(np.int32)
    a, rn = oracle.assign(N, g, E, tabs, topk, src, seed=seed, step=seed, mode=0)
    assert a.tolist() == rows[:, 4:6].tolist()
    assert rn.tolist() == rows[:, 6].tolist()
    o, orn = oracle.assign(N, g, E, tabs, topk, src, mode=1)
    assert o.tolist() == rows[:, 7:9].tolist()
    assert orn.tolist() == rows[:, 9].tolist()
    Va, ca, _ = oracle.traffic(a, N, g, src)
    Vo, co, _ = oracle.traffic(o, N, g, src)
    assert [Va, Vo] == fig1["V"]
    assert [ca, co] == fig1["cross"]


def test_layout_tables_reject_invalid(fig1):
    N, g, E = fig1["N"], fig1["g"], fig1["E"]
    t = fig1["table"].copy()
    t[3, 0] = -1  # d loses its only replica: coverage (Eq. 2) fails
    with pytest.raises(oracle.OracleError):
        oracle.layout_tables(N, g, E, t)
    t = fig1["table"].copy()
    t[0, 1] = 0  # a twice on GPU0
    with pytest.raises(oracle.OracleError):
        oracle.layout_tables(N, g, E, t)
    with pytest.raises(oracle.OracleError):  # owner of b does not hold b
        oracle.layout_tables(N, g, E, fig1["table"], np.array([0, 1, 1, 3], np.int32))
    t = fig1["table"].copy()
    t[0, 1] = 4  # id outside [0, E)
    with pytest.raises(oracle.OracleError):
        oracle.layout_tables(N, g, E, t)


# ------------------------------------------------------- brute force covers
def _random_layout(rng, N, g, E, S):
    """Every expert once on a random rank with room, then random extra
    replicas (no expert twice on a rank). Needs G*S >= E."""
    G = N * g
    assert G * S >= E
    slots = [[] for _ in range(G)]
    for e in rng.permutation(E):
        free = [r for r in range(G) if len(slots[r]) < S]
        slots[free[rng.integers(len(free))]].append(int(e))
    for _ in range(int(rng.integers(0, G * S - E + 1))):
        e = int(rng.integers(E))
        free = [r for r in range(G) if len(slots[r]) < S and e not in slots[r]]
        if free:
            slots[free[rng.integers(len(free))]].append(e)
    table = np.full((G, S), -1, np.int32)
    for r in range(G):
        table[r, : len(slots[r])] = slots[r]
    return table


def _brute_min_cover(D, src, table, g):
    """Over every choice of a holding rank per selected expert: the minimum
    number of distinct remote nodes, and the remote-node bitmasks reaching it."""
    home = src // g
    holders = [[r for r in range(table.shape[0]) if e in table[r]] for e in D]
    best, masks = None, set()
    for choice in itertools.product(*holders):
        m = 0
        for r in choice:
            if r // g != home:
                m |= 1 << (r // g)
        c = popcount(m)
        if best is None or c < best:
            best, masks = c, {m}
        elif c == best:
            masks.add(m)
    return best, masks


@pytest.mark.parametrize("case", range(40))
def test_brute_force_min_cover(case):
    rng = np.random.default_rng(1000 + case)
    N = int(rng.integers(2, 6))
    g = int(rng.integers(1, 4))
    E = int(rng.integers(2, 9))
    K = int(rng.integers(1, min(4, E) + 1))
    S = int(rng.integers(-(-E // (N * g)), 4 + -(-E // (N * g))))
    table = _random_layout(rng, N, g, E, S)
    G = N * g
    T = 48
    topk = np.stack([rng.choice(E, size=K, replace=False) for _ in range(T)]).astype(np.int32)
    src = np.sort(rng.integers(0, G, size=T)).astype(np.int32)
    tabs = oracle.layout_tables(N, g, E, table)
    a, rn = oracle.assign(N, g, E, tabs, topk, src, seed=case, step=1)
    nm = tabs[0]
    for t in range(T):
        best, masks = _brute_min_cover(topk[t], src[t], table, g)
        home = src[t] // g
        assert popcount(rn[t]) == best
        assert int(rn[t]) == min(masks)  # smallest node-id bitmask among minimum covers
        got = 0
        for j in range(K):
            r = a[t, j]
            assert 0 <= r < G and topk[t, j] in table[r]  # e in P_{r_te} (Eq. 2)
            if nm[topk[t, j]] >> home & 1:
                assert r // g == home  # experts held locally run locally
            if r // g != home:
                got |= 1 << (r // g)
        assert got == int(rn[t])  # each chosen remote node is used
    V, _, _ = oracle.traffic(a, N, g, src)
    assert V == sum(popcount(v) for v in rn)


# ------------------------------------------------------------ special cases
def test_no_replicas_equals_owner_only():
    w = W.with_sizes(W.WORKLOADS["tiny"], T=2048)
    table, owner = W.layout(w, 0, S=w.E // w.G, replicas="none")  # literal S = 2
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    topk, _ = W.routing(w, 0)
    a, rn = oracle.assign(w.N, w.g, w.E, tabs, topk.numpy(), seed=4)
    o, orn = oracle.assign(w.N, w.g, w.E, tabs, topk.numpy(), mode=1)
    assert np.array_equal(a, o) and np.array_equal(rn, orn)


def test_single_node_everything_local():
    rng = np.random.default_rng(3)
    N, g, E, K = 1, 4, 8, 3
    table = _random_layout(rng, N, g, E, 4)
    tabs = oracle.layout_tables(N, g, E, table)
    topk = np.stack([rng.choice(E, size=K, replace=False) for _ in range(64)]).astype(np.int32)
    a, rn = oracle.assign(N, g, E, tabs, topk)
    assert np.all(rn == 0)
    for t in range(64):
        for j in range(K):
            assert topk[t, j] in table[a[t, j]]


def test_every_expert_local_means_no_remote_nodes():
    N, g, E = 4, 2, 6
    table = np.tile(np.arange(E, dtype=np.int32)[None, :], (N * g, 1))  # all experts on every rank
    tabs = oracle.layout_tables(N, g, E, table)
    rng = np.random.default_rng(8)
    topk = np.stack([rng.choice(E, size=3, replace=False) for _ in range(400)]).astype(np.int32)
    src = np.sort(rng.integers(0, N * g, size=400)).astype(np.int32)
    a, rn = oracle.assign(N, g, E, tabs, topk, src)
    assert np.all(rn == 0)
    assert np.all(a // g == (src // g)[:, None])


def test_k1_single_selection():
    w = W.with_sizes(W.WORKLOADS["clusters-e64"], T=512, K=1)
    table, owner = W.layout(w, 1)
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    topk, _ = W.routing(w, 1)
    a, rn = oracle.assign(w.N, w.g, w.E, tabs, topk.numpy())
    assert np.all(np.array([popcount(v) for v in rn]) <= 1)


# ---------------------------------------------------------- uniform draws
def test_rank_choice_uniform_within_node():
    """UniformChoice: an expert held by 3 ranks of the source node."""
    N, g, E = 2, 4, 2
    table = np.array([[0, 1], [0, -1], [0, -1], [-1, -1],
                      [1, -1], [-1, -1], [-1, -1], [-1, -1]], np.int32)
    tabs = oracle.layout_tables(N, g, E, table)
    T = 300000  # 10^5 per candidate rank
    topk = np.zeros((T, 1), np.int32)
    src = np.full(T, 3, np.int32)
    a, _ = oracle.assign(N, g, E, tabs, topk, src, seed=11)
    cnt = np.bincount(a.ravel(), minlength=8)
    assert cnt[[3, 4, 5, 6, 7]].sum() == 0
    _, pval = chisquare(cnt[:3])
    assert pval > 1e-4


def test_node_choice_uniform_within_cover():
    """RandomNode: U = {e1 on node 1, e2 on node 2, e3 on nodes 1 and 2}; the
    cover is {1, 2} and e3 must land on either node with equal odds."""
    N, g, E = 3, 1, 3
    table = np.array([[-1, -1], [0, 2], [1, 2]], np.int32)
    tabs = oracle.layout_tables(N, g, E, table)
    T = 200000  # 10^5 per candidate node
    topk = np.tile(np.array([[0, 1, 2]], np.int32), (T, 1))
    src = np.zeros(T, np.int32)
    a, rn = oracle.assign(N, g, E, tabs, topk, src, seed=5, step=2)
    assert np.all(rn == 0b110)
    assert np.all(a[:, 0] == 1) and np.all(a[:, 1] == 2)
    _, pval = chisquare(np.bincount(a[:, 2], minlength=3)[1:])
    assert pval > 1e-4


def test_deterministic_and_seed_dependent():
    w = W.with_sizes(W.WORKLOADS["clusters-e64"], T=4096)
    table, owner = W.layout(w, 1)
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    topk = W.routing(w, 1)[0].numpy()
    a1, _ = oracle.assign(w.N, w.g, w.E, tabs, topk, seed=1, step=0)
    a2, _ = oracle.assign(w.N, w.g, w.E, tabs, topk, seed=1, step=0)
    a3, _ = oracle.assign(w.N, w.g, w.E, tabs, topk, seed=1, step=1)
    assert np.array_equal(a1, a2)
    assert not np.array_equal(a1, a3)


# ------------------------------------------------ workloads at reduced size
@pytest.mark.parametrize("name", ["tiny", "clusters-e64", "colocate-e128", "colocate-e256", "drift-e384"])
def test_reduced_configs_valid_and_never_worse_than_owner_only(name):
    w = W.with_sizes(W.WORKLOADS[name], T=W.WORKLOADS[name].G * 16)
    table, owner = W.layout(w, w.seed)
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    topk = W.routing(w, w.seed)[0].numpy()
    a, rn = oracle.assign(w.N, w.g, w.E, tabs, topk, seed=w.seed)
    o, orn = oracle.assign(w.N, w.g, w.E, tabs, topk, mode=1)
    held = [set(table[r][table[r] >= 0].tolist()) for r in range(w.G)]
    assert all(topk[t, j] in held[a[t, j]] for t in range(w.T) for j in range(w.K))
    pa = np.array([popcount(v) for v in rn])
    po = np.array([popcount(v) for v in orn])
    assert np.all(pa <= po)  # Algorithm 1's cover is minimal per token
