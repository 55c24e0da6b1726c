"""The seeded generator: shapes, determinism, layout validity (Eq. 2's
coverage and slot budget) and the planted structure."""
import numpy as np
import pytest

import oracle
from paper_2609_36959_amd import workload as W


@pytest.mark.parametrize("name", ["tiny", "clusters-e64", "colocate-e128", "colocate-e256", "drift-e384"])
def test_layout_valid(name):
    w = W.WORKLOADS[name]
    table, owner = W.layout(w, w.seed)
    assert table.shape == (w.G, w.S)
    nm, rm, own = oracle.layout_tables(w.N, w.g, w.E, table, owner)  # raises if invalid
    assert np.all(own == owner)
    reps = np.array([sum(bin(int(v)).count("1") for v in rm[e]) for e in range(w.E)])
    assert reps.min() >= 1 and reps.sum() == np.count_nonzero(table >= 0)
    if w.replicas == "intra_node_top":
        assert np.all(np.array([bin(int(v)).count("1") for v in nm]) == 1)  # co-located
        assert (reps > 1).sum() == round(w.top_frac * w.E)
    else:
        assert reps.sum() == w.G * w.S


def test_routing_deterministic_and_shaped():
    w = W.with_sizes(W.WORKLOADS["colocate-e128"], T=1000)
    a, g = W.routing(w, 2)
    b, h = W.routing(w, 2)
    assert a.shape == (1000, w.K) and a.dtype.is_floating_point is False
    assert np.array_equal(a.numpy(), b.numpy()) and np.array_equal(g.numpy(), h.numpy())
    srt = np.sort(a.numpy(), axis=1)
    assert np.all(np.diff(srt, axis=1) > 0)  # distinct experts per token
    assert np.allclose(g.numpy().sum(1), 1.0, atol=1e-6)
    assert np.all(np.diff(g.numpy(), axis=1) <= 0)  # slot j is the j-th largest


def test_planted_clusters_co_activate():
    w = W.with_sizes(W.WORKLOADS["clusters-e64"], T=4096)
    topk = W.routing(w, 1)[0].numpy()
    C, cnt = oracle.coact_stats(topk, w.E)
    cl = W.clusters(w, 1)
    same = np.zeros((w.E, w.E), bool)
    for c in cl:
        same[np.ix_(c, c)] = True
    np.fill_diagonal(same, False)
    assert C[same].mean() > 3 * C[~same & ~np.eye(w.E, dtype=bool)].mean()


def test_drift_moves_bias_and_hot_order():
    w = W.WORKLOADS["drift-e384"]
    b0, b8 = W.bias(w, 4, 0), W.bias(w, 4, 8)
    assert np.array_equal(np.sort(b0), np.sort(b8)) and not np.array_equal(b0, b8)
    t1, _ = W.layout(w, 4)
    t2, _ = W.layout(w, 4, hot_order=np.argsort(-b8, kind="stable"), plan=8)
    assert not np.array_equal(t1, t2)
