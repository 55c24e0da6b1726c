"""Pins of the oracle's combine (gate-weighted sum back to token order,
Fig. 1's last stage): an fp64 sum within the error bound of an fp32
fused-multiply-add chain, the dispatch/combine round trip, and K = 1."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36959_amd import workload as W

U32 = 2.0**-24


def _bits(t):
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def _widen(bits):
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()


@pytest.mark.parametrize("T,K,d", [(64, 8, 96), (33, 6, 40), (5, 1, 8), (17, 2, 512)])
def test_fp64_bound(T, K, d):
    rng = np.random.default_rng(T + K + d)
    eo = _bits(torch.randn(T * K, d).to(torch.bfloat16))
    pos = rng.permutation(T * K).reshape(T, K).astype(np.int32)
    gates = rng.standard_normal((T, K)).astype(np.float32)
    y, y32 = oracle.combine(eo, pos, gates)
    v = _widen(eo)[pos]                                   # [T, K, d]
    terms = gates.astype(np.float64)[:, :, None] * v
    exact = terms.sum(1)
    gamma = K * U32 / (1 - K * U32)
    assert np.all(np.abs(y32.astype(np.float64) - exact) <= gamma * np.abs(terms).sum(1) + 1e-45)
    # the bf16 output is the round-to-nearest-even narrowing of the fp32 sum
    want = _bits(torch.from_numpy(y32).to(torch.bfloat16))
    assert np.array_equal(y, want)


@pytest.mark.parametrize("name", ["tiny", "clusters-e64", "colocate-e256"])
def test_round_trip_identity(name):
    """expert_out = packed and gates summing to one give back x (by value)."""
    w = W.with_sizes(W.WORKLOADS[name], T=W.WORKLOADS[name].G * 8, d=64)
    table, owner = W.layout(w, w.seed)
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    topk, gates = W.routing(w, w.seed)
    a, _ = oracle.assign(w.N, w.g, w.E, tabs, topk.numpy(), seed=w.seed)
    x = _bits(W.hidden(w, w.seed))
    _, _, pos, packed = oracle.dispatch(a, w.G, None, x)
    y, _ = oracle.combine(packed, pos, gates.numpy())
    assert np.array_equal(_widen(y), _widen(x))


def test_k1_unit_gate_is_a_gather():
    rng = np.random.default_rng(2)
    eo = _bits(torch.randn(40, 24).to(torch.bfloat16))
    pos = rng.integers(0, 40, size=(30, 1)).astype(np.int32)
    y, _ = oracle.combine(eo, pos, np.ones((30, 1), np.float32))
    assert np.array_equal(_widen(y), _widen(eo)[pos[:, 0]])
