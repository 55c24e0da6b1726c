"""Pins of the oracle's node-deduplicated dispatch layout: one row per
(token, destination node), grouped by (source rank, destination node),
stable in the token index, with a forwarding mask of the node's ranks."""
import numpy as np
import pytest

import oracle
from conftest import read_golden
from paper_2609_36959_amd import workload as W


def _golden():
    return {f[0]: [int(v) for v in f[1:]] for f in read_golden("fig1_node_dispatch.txt")}


def _sorted_layout(assigned, src, N, g):
    """The same layout from its definition as a sort: the items (s_t, n, t)
    for every distinct destination node n of token t, sorted
    lexicographically, are the packed rows in order."""
    T, K = assigned.shape
    items = []
    for t in range(T):
        masks = {}
        for r in assigned[t]:
            masks[int(r) // g] = masks.get(int(r) // g, 0) | (1 << (int(r) % g))
        for n, m in masks.items():
            items.append((int(src[t]), n, t, m))
    items.sort()
    node_pos = np.full((T, N), -1, np.int64)
    fwd = np.array([m for _, _, _, m in items], np.uint32)
    tok = np.array([t for _, _, t, _ in items], np.int64)
    for row, (_, n, t, _) in enumerate(items):
        node_pos[t, n] = row
    counts = np.zeros((N * g, N), np.int64)
    for s, n, _, _ in items:
        counts[s, n] += 1
    return counts, node_pos, fwd, tok


def _eq1_traffic(assigned, src, g):
    """V of Eq. 1: distinct destination nodes other than the source's."""
    return sum(len({int(r) // g for r in assigned[t]} - {int(src[t]) // g})
               for t in range(assigned.shape[0]))


@pytest.mark.parametrize("which,cols", [("alg1", (4, 6)), ("owner", (7, 9))])
def test_fig1_worked_example(fig1, which, cols):
    gold = _golden()
    rows = np.array(fig1["tokens"], np.int64)
    src = rows[:, 1].astype(np.int32)
    assigned = rows[:, cols[0]:cols[1]].astype(np.int32)
    counts, offsets, node_pos, fwd, tok, _ = oracle.node_dispatch(assigned, 2, 2, src)
    assert node_pos.ravel().tolist() == gold[f"{which}_node_pos"]
    assert offsets.tolist() == gold[f"{which}_offsets"]
    assert fwd.tolist() == gold[f"{which}_fwd"]
    assert tok.tolist() == gold[f"{which}_row_token"]
    cross = sum(1 for t in range(4) for n in range(2) if node_pos[t, n] >= 0 and n != src[t] // 2)
    assert cross == gold[f"{which}_cross_rows"][0]


@pytest.mark.parametrize("N,g,T,K,ragged", [(2, 4, 257, 2, True), (4, 8, 512, 8, False),
                                            (8, 2, 300, 5, True), (1, 4, 64, 3, False),
                                            (16, 1, 96, 16, True)])
def test_matches_sorted_definition(N, g, T, K, ragged):
    rng = np.random.default_rng(N * 131 + g * 7 + T)
    G = N * g
    src = W.ragged_src(T, G, seed=T) if ragged else W.contiguous_src(T, G)
    assigned = rng.integers(0, G, size=(T, K)).astype(np.int32)
    x = rng.integers(0, 2**16, size=(T, 8)).astype(np.uint16)
    counts, offsets, node_pos, fwd, tok, packed = oracle.node_dispatch(assigned, N, g, src, x)
    c2, p2, f2, t2 = _sorted_layout(assigned, src, N, g)
    assert np.array_equal(counts, c2)
    assert np.array_equal(offsets, np.concatenate([[0], np.cumsum(c2.ravel())]))
    assert np.array_equal(node_pos, p2)
    assert np.array_equal(fwd, f2)
    assert np.array_equal(tok, t2)
    assert np.array_equal(packed, x[t2])
    if not ragged:
        r_null = oracle.node_dispatch(assigned, N, g, None)
        assert np.array_equal(r_null[2], node_pos)


def test_one_rank_per_node_reduces_to_pair_dispatch():
    """With g = 1 and K distinct ranks per token, every pair is its own node
    row and buckets (s, n) are buckets (s, r): the node layout is the
    per-pair layout, row for row."""
    rng = np.random.default_rng(5)
    G, T, K = 16, 640, 6
    src = W.ragged_src(T, G, seed=11)
    assigned = np.stack([rng.permutation(G)[:K] for _ in range(T)]).astype(np.int32)
    x = rng.integers(0, 2**16, size=(T, 8)).astype(np.uint16)
    counts, offsets, pos, packed = oracle.dispatch(assigned, G, src, x)
    nc, no, node_pos, fwd, tok, npacked = oracle.node_dispatch(assigned, G, 1, src, x)
    assert np.array_equal(nc, counts)
    assert np.array_equal(no, offsets)
    assert np.array_equal(np.take_along_axis(node_pos, assigned.astype(np.int64), 1), pos)
    assert np.all(fwd == 1)
    assert np.array_equal(npacked, packed)


def test_invariants_on_reduced_workload():
    w = W.with_sizes(W.WORKLOADS["colocate-e256"], T=4096)
    table, owner = W.layout(w, 3)
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    topk = W.routing(w, 3)[0].numpy()
    src = W.contiguous_src(w.T, w.G)
    for mode in (0, 1):
        a, rn = oracle.assign(w.N, w.g, w.E, tabs, topk, seed=3, mode=mode)
        counts, offsets, node_pos, fwd, tok, _ = oracle.node_dispatch(a, w.N, w.g)
        node = a // w.g
        distinct_nodes = np.array([len(set(r)) for r in node])
        distinct_ranks = np.array([len(set(r)) for r in a])
        assert offsets[-1] == distinct_nodes.sum() == (node_pos >= 0).sum()
        assert np.array_equal(np.sort(node_pos[node_pos >= 0]), np.arange(offsets[-1]))
        # forwarding masks deliver every distinct (token, rank) exactly once
        assert sum(bin(int(m)).count("1") for m in fwd) == distinct_ranks.sum()
        for t in range(0, w.T, 97):
            for j in range(w.K):
                row = node_pos[t, node[t, j]]
                assert row >= 0 and tok[row] == t
                assert (int(fwd[row]) >> (int(a[t, j]) % w.g)) & 1
        # rows crossing nodes are Eq. 1's V, and match Algorithm 1's b*
        home = src // w.g
        cross = sum(int((node_pos[t] >= 0).sum()) - int(node_pos[t, home[t]] >= 0)
                    for t in range(w.T))
        assert cross == _eq1_traffic(a, src, w.g)
        if mode == 0:
            assert cross == sum(bin(int(v)).count("1") for v in rn)
        # every row lies in its (source, node) bucket, increasing in t
        row_bucket = np.searchsorted(offsets, np.arange(offsets[-1]), side="right") - 1
        s_of_row, n_of_row = row_bucket // w.N, row_bucket % w.N
        assert np.array_equal(s_of_row, src[tok])
        assert np.all(node_pos[tok, n_of_row] == np.arange(offsets[-1]))
        same = row_bucket[1:] == row_bucket[:-1]
        assert np.all(tok[1:][same] > tok[:-1][same])


def test_empty_and_errors():
    counts, offsets, node_pos, fwd, tok, _ = oracle.node_dispatch(
        np.zeros((0, 4), np.int32), 2, 2, np.zeros(0, np.int32))
    assert offsets.tolist() == [0] * 9 and node_pos.shape == (0, 2) and fwd.size == 0
    with pytest.raises(oracle.OracleError):
        oracle.node_dispatch(np.array([[0, 4]], np.int32), 2, 2, np.array([0], np.int32))
    with pytest.raises(oracle.OracleError):
        oracle.node_dispatch(np.array([[0, 1]], np.int32), 2, 2, np.array([4], np.int32))
