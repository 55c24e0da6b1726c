"""Pins of the oracle's co-activation statistics (Section 3.2, Stage 1:
c_ij counts tokens selecting both i and j, w_e counts tasks of e)."""
import numpy as np
import pytest

import oracle
from paper_2609_36959_amd import workload as W


def _distinct_topk(rng, T, E, K):
    return np.stack([rng.choice(E, size=K, replace=False) for _ in range(T)]).astype(np.int32)


def test_fig1_tokens(fig1):
    topk = np.array([[t[2], t[3]] for t in fig1["tokens"]], np.int32)
    C, cnt = oracle.coact_stats(topk, fig1["E"])
    want = np.zeros((4, 4), np.uint32)
    for i, j, c in fig1["coact"]:
        want[i, j] = c
    assert np.array_equal(C, want)
    assert cnt.tolist() == fig1["count"]


@pytest.mark.parametrize("T,E,K", [(1, 5, 1), (300, 12, 4), (257, 33, 7), (64, 8, 8)])
def test_brute_force_gram_matrix(T, E, K):
    """With distinct selections per token, C = A^T A - diag(A^T A) where A is
    the T x E 0/1 selection matrix, and count = column sums of A."""
    rng = np.random.default_rng(T * 1000 + E)
    topk = _distinct_topk(rng, T, E, K)
    A = np.zeros((T, E), np.int64)
    A[np.arange(T)[:, None], topk] = 1
    gram = A.T @ A
    C, cnt = oracle.coact_stats(topk, E)
    assert np.array_equal(C.astype(np.int64), gram - np.diag(np.diag(gram)))
    assert np.array_equal(cnt.astype(np.int64), A.sum(0))


@pytest.mark.parametrize("name", ["tiny", "clusters-e64", "colocate-e128", "colocate-e256", "drift-e384"])
def test_invariants_reduced_configs(name):
    w = W.with_sizes(W.WORKLOADS[name], T=2048)
    topk, _ = W.routing(w, seed=w.seed)
    C, cnt = oracle.coact_stats(topk.numpy(), w.E)
    C = C.astype(np.int64)
    assert np.array_equal(C, C.T)
    assert np.all(np.diag(C) == 0)
    assert np.array_equal(C.sum(1), (w.K - 1) * cnt.astype(np.int64))
    assert cnt.sum() == w.T * w.K
    assert C.sum() == w.T * w.K * (w.K - 1)


def test_accumulates_across_calls():
    rng = np.random.default_rng(5)
    a = _distinct_topk(rng, 100, 10, 3)
    b = _distinct_topk(rng, 77, 10, 3)
    C, cnt = oracle.coact_stats(a, 10)
    C, cnt = oracle.coact_stats(b, 10, C, cnt)
    C2, cnt2 = oracle.coact_stats(np.concatenate([a, b]), 10)
    assert np.array_equal(C, C2) and np.array_equal(cnt, cnt2)


def test_rejects_out_of_range_ids():
    with pytest.raises(oracle.OracleError):
        oracle.coact_stats(np.array([[0, 9]], np.int32), 9)


def test_repeated_ids_follow_the_ordered_slot_pair_definition():
    """A token that holds an expert m times: every ordered pair of distinct
    slots counts, so the diagonal entry gets m(m - 1) and a pair (i, j) the
    product of the multiplicities. Counted here by hand on worked tokens."""
    E = 6
    topk = np.array([[2, 2, 2, 5],      # 2 three times: C[2][2] += 6; (2, 5) += 3 each way
                     [1, 1, 4, 4],      # C[1][1] += 2, C[4][4] += 2; (1, 4) += 4 each way
                     [0, 3, 3, 0]],     # C[0][0] += 2, C[3][3] += 2; (0, 3) += 4 each way
                    np.int32)
    C, cnt = oracle.coact_stats(topk, E)
    want = np.zeros((E, E), np.uint32)
    for i, j, v in [(2, 2, 6), (2, 5, 3), (5, 2, 3), (1, 1, 2), (4, 4, 2), (1, 4, 4), (4, 1, 4),
                    (0, 0, 2), (3, 3, 2), (0, 3, 4), (3, 0, 4)]:
        want[i, j] += v
    assert np.array_equal(C, want)
    assert cnt.tolist() == [2, 2, 3, 2, 2, 1]
    # row sums stay (K - 1) * count with the diagonal included
    assert np.array_equal(C.sum(1), 3 * cnt)
