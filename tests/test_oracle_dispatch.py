"""Pins of the oracle's dispatch layout: buckets (source, destination) in
row-major order, stable in the pair index, one packed row per pair."""
import numpy as np
import pytest

import oracle
from paper_2609_36959_amd import workload as W


def _library_layout(assigned, src, G):
    """The same layout from library primitives: a stable sort of the pairs
    by bucket key gives the packed order; pos is its inverse permutation."""
    T, K = assigned.shape
    key = (np.repeat(src.astype(np.int64), K) * G + assigned.ravel()).astype(np.int64)
    order = np.argsort(key, kind="stable")
    pos = np.empty(T * K, np.int64)
    pos[order] = np.arange(T * K)
    counts = np.bincount(key, minlength=G * G).reshape(G, G)
    offsets = np.concatenate([[0], np.cumsum(counts.ravel())])
    return counts, offsets, pos.reshape(T, K)


def test_fig1_pos_and_offsets(fig1):
    rows = np.array(fig1["tokens"], np.int64)
    src = rows[:, 1].astype(np.int32)
    assigned = rows[:, 4:6].astype(np.int32)
    counts, offsets, pos, _ = oracle.dispatch(assigned, 4, src)
    assert pos.ravel().tolist() == fig1["pos"]
    assert offsets.tolist() == fig1["offsets"]
    assert counts.sum() == 8


@pytest.mark.parametrize("G,T,K,ragged", [(8, 512, 2, False), (4, 301, 3, True),
                                          (16, 1024, 8, True), (1, 10, 4, False)])
def test_matches_stable_sort(G, T, K, ragged):
    rng = np.random.default_rng(G * 7 + T)
    if ragged:
        src = W.ragged_src(T, G, seed=T)
    else:
        src = W.contiguous_src(T, G)
    assigned = rng.integers(0, G, size=(T, K)).astype(np.int32)
    d = 16
    x = rng.integers(0, 2**16, size=(T, d)).astype(np.uint16)
    counts, offsets, pos, packed = oracle.dispatch(assigned, G, src, x)
    c2, o2, p2 = _library_layout(assigned, src, G)
    assert np.array_equal(counts, c2)
    assert np.array_equal(offsets, o2)
    assert np.array_equal(pos, p2)
    assert np.array_equal(packed[pos.ravel()], np.repeat(x, K, axis=0))
    assert np.array_equal(counts.sum(1), np.bincount(src, minlength=G) * K)  # row sums
    if not ragged:
        _, _, pos_null, _ = oracle.dispatch(assigned, G, None)
        assert np.array_equal(pos_null, pos)


def test_invariants_on_reduced_config():
    w = W.with_sizes(W.WORKLOADS["colocate-e256"], T=4096)
    table, owner = W.layout(w, 3)
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    topk = W.routing(w, 3)[0].numpy()
    a, _ = oracle.assign(w.N, w.g, w.E, tabs, topk, seed=3)
    counts, offsets, pos, _ = oracle.dispatch(a, w.G)
    assert offsets[-1] == w.T * w.K == counts.sum()
    assert np.array_equal(np.sort(pos.ravel()), np.arange(w.T * w.K))  # a permutation
    assert np.array_equal(counts.sum(0), np.bincount(a.ravel(), minlength=w.G))  # rank loads
    src = W.contiguous_src(w.T, w.G)
    bucket = np.searchsorted(offsets, pos.ravel(), side="right") - 1
    assert np.array_equal(bucket, np.repeat(src, w.K) * w.G + a.ravel())
    # stability: inside each bucket pos increases with the pair index
    order = np.argsort(pos.ravel())          # pair index held by each packed row
    same = bucket[order][1:] == bucket[order][:-1]
    assert np.all(order[1:][same] > order[:-1][same])


def test_rejects_bad_ranks():
    with pytest.raises(oracle.OracleError):
        oracle.dispatch(np.array([[0, 4]], np.int32), 4, np.array([0], np.int32))
