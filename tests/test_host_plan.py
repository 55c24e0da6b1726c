"""The library's host-side Stage-1 planner (cobalt_plan_layout) against the
oracle, on the CPU: identical slot tables, owners, planned work, objective
and feasibility, on the workloads' own statistics, random instances and the
structured cases of the oracle's pins."""
import itertools

import numpy as np
import pytest

import oracle
from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import workload as W


def same(N, g, E, S, c, w, eps):
    a = B.cobalt_plan_layout(N, g, E, S, c, w, eps)
    b = oracle.plan_layout(N, g, E, S, c, w, eps)
    for x, y in zip(a[:3], b[:3]):
        assert np.array_equal(x, y)
    assert a[3] == b[3] and a[4] == b[4]
    return a


@pytest.mark.parametrize("name", W.NAMES)
def test_workload_statistics(name):
    """The counts of a reduced step of each workload, as the EMA after its
    first update would hold them."""
    w = W.with_sizes(W.WORKLOADS[name], T=min(W.WORKLOADS[name].T, 8192))
    topk = W.routing(w, w.seed)[0].numpy()
    C, n = oracle.coact_stats(topk, w.E)
    for eps in (0.15, 0.0, 0.5):
        same(w.N, w.g, w.E, w.S, C.astype(np.float32), n.astype(np.float32), eps)


@pytest.mark.parametrize("N,g,E,S", [(2, 2, 16, 6), (4, 2, 24, 4), (8, 4, 96, 5), (3, 3, 40, 6),
                                     (16, 1, 16, 2), (1, 8, 32, 5), (4, 8, 64, 3)])
def test_random_instances(N, g, E, S):
    rng = np.random.default_rng(N * 31 + E)
    for trial in range(4):
        c = rng.random((E, E)) * 100
        c[rng.random((E, E)) > 0.5] = 0
        c = np.triu(c, 1)
        c = (c + c.T).astype(np.float32)
        w = (rng.pareto(1.2, E) * 100 + 1).astype(np.float32)
        if trial == 3:
            w = np.round(w / 50).astype(np.float32)  # many ties, some zeros
        same(N, g, E, S, c, w, 0.15)


def test_structured_cases():
    rng = np.random.default_rng(7)
    E = 24
    groups = rng.permutation(E).reshape(4, 6)
    c = np.zeros((E, E), np.float32)
    for grp in groups:
        for a, b in itertools.permutations(grp, 2):
            c[a, b] = 10.0
    out = same(4, 2, E, 3, c, np.ones(E, np.float32), 0.15)
    assert out[3] == 600.0
    w = np.ones(16, np.float32)
    w[5] = 20.0
    same(4, 2, 16, 4, np.zeros((16, 16), np.float32), w, 0.15)
    same(2, 2, 8, 2, np.zeros((8, 8), np.float32), np.zeros(8, np.float32), 0.15)
    c = np.zeros((4, 4), np.float32)
    c[0, 1] = c[1, 0] = 100.0
    assert same(2, 1, 4, 2, c, np.array([3, 3, 1, 1], np.float32), 0.15)[4]


def test_library_rejects_what_the_oracle_rejects():
    z = np.zeros((8, 8), np.float32)
    one = np.ones(8, np.float32)
    bad = z.copy()
    bad[0, 1] = np.nan
    huge = z.copy()
    huge[0, 1] = 2.0**29
    for args in ((2, 2, 8, 1, z, one, 0.1),             # G*S < E
                 (2, 2, 8, 2, bad, one, 0.1),           # NaN pair weight
                 (2, 2, 8, 2, huge, one, 0.1),          # pair weight above 2^28
                 (2, 2, 8, 2, z, -one, 0.1),            # negative workload
                 (2, 2, 8, 2, z, one, -1.0)):           # negative eps
        with pytest.raises(B.CobaltError):
            B.cobalt_plan_layout(*args)
        with pytest.raises(oracle.OracleError):
            oracle.plan_layout(*args)
    # the largest pair weight accepted: both plan it, identically
    edge = z.copy()
    edge[0, 1] = edge[1, 0] = 2.0**28
    same(2, 2, 8, 2, edge, one, 0.1)


def tight_instance(seed):
    """Zipf(1.2) work on 4 x 4 ranks with one spare slot per rank: the node
    fill of step 1 leaves ranks above the cap that only the repair across
    nodes can bring back."""
    rng = np.random.default_rng(100 + seed)
    N, g = 4, 4
    E = 48 + 8 * (seed % 3)
    S = -(-E // (N * g)) + 1
    w = ((1.0 / np.arange(1, E + 1) ** 1.2)[rng.permutation(E)] * 1000).astype(np.float32)
    c = (rng.random((E, E)) * 10).astype(np.float32)
    c[rng.random((E, E)) > 0.3] = 0
    c = np.triu(c, 1)
    return N, g, E, S, c + c.T, w


@pytest.mark.parametrize("seed", range(12))
def test_tight_slots_and_the_repair_across_nodes(seed):
    N, g, E, S, c, w = tight_instance(seed)
    same(N, g, E, S, c, w, 0.15)
