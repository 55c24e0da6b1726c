"""The library's host-side Stage-2 rebalancing (cobalt_intra_node_rebalance)
against the oracle, on the CPU: identical tables, owners and rank loads."""
import numpy as np
import pytest

import oracle
from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import workload as W


@pytest.mark.parametrize("name", W.NAMES)
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_library_matches_oracle(name, seed):
    w = W.WORKLOADS[name]
    table, owner = W.layout(w, w.seed)
    rng = np.random.default_rng(seed)
    load = rng.gamma(0.7, 50.0, size=(w.E, w.G)).astype(np.float32)
    load[rng.random(load.shape) < 0.2] = 0.0  # ties
    load[:, : w.g] = np.round(load[:, : w.g])  # more ties
    for own in (owner, None):
        a = B.cobalt_intra_node_rebalance(w.N, w.g, w.E, table.shape[1], table, own, load)
        b = oracle.intra_node_rebalance(w.N, w.g, w.E, table, own, load)
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


def test_library_rejects_what_the_oracle_rejects():
    table = np.array([[0], [1]], np.int32)
    load = np.ones((2, 2), np.float32)
    load[1, 1] = np.inf
    with pytest.raises(B.CobaltError):
        B.cobalt_intra_node_rebalance(1, 2, 2, 1, table, None, load)
    with pytest.raises(oracle.OracleError):
        oracle.intra_node_rebalance(1, 2, 2, table, None, load)
    bad = np.array([[0], [0]], np.int32)  # expert 1 uncovered
    with pytest.raises(B.CobaltError):
        B.cobalt_intra_node_rebalance(1, 2, 2, 1, bad, None, np.ones((2, 2), np.float32))
