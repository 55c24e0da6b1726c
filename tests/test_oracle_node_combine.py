"""Pins of the oracle's node-level combine (the reverse of the
node-deduplicated dispatch, Section 1 and Section 3.1): partial sums per
(token, node) rounded to bf16, then summed at the source in node order.

The pins are the reduction to the plain combine on one node; exact
arithmetic (power-of-two gates, small-integer values: every partial and
every sum is exact, so the result is the exact sum whatever the rounding
order); two cases worked by hand that fix the two roundings and the order
of the source sum; the skip rules; and the error bound against the plain
combine on random data."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36959_amd import workload as W


def _bits(t):
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def _widen(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).double().numpy()


def _bf16(values):
    """bf16 bits of values that bf16 represents exactly."""
    v = np.asarray(values, np.float32)
    u = v.view(np.uint32)
    assert np.all(u & 0xFFFF == 0), "not exactly representable"
    return (u >> 16).astype(np.uint16)


def _layout(assigned, N, g):
    src = np.zeros(len(assigned), np.int32)
    return oracle.node_dispatch(assigned, N, g, src=src)[2]


@pytest.mark.parametrize("T,K,g,d", [(40, 8, 8, 64), (13, 3, 2, 24), (9, 1, 4, 8)])
def test_single_node_equals_the_plain_combine(T, K, g, d):
    """With one node the only partial of a token is the plain combine's fp32
    sum rounded to bf16, and the source adds it to 0: y is the plain
    combine's result bit for bit, and so is the partial row."""
    rng = np.random.default_rng(T * K + g)
    a = rng.integers(0, g, size=(T, K)).astype(np.int32)
    pos = rng.permutation(T * K).reshape(T, K).astype(np.int32)
    eo = _bits(torch.randn(T * K, d).to(torch.bfloat16))
    gates = rng.standard_normal((T, K)).astype(np.float32)
    node_pos = _layout(a, 1, g)
    part, y = oracle.node_combine(eo, pos, a, gates, node_pos, g)
    flat, _ = oracle.combine(eo, pos, gates)
    assert np.array_equal(y, flat)
    assert np.array_equal(part[node_pos[:, 0]], flat)


@pytest.mark.parametrize("N,g,K", [(4, 2, 8), (8, 8, 8), (3, 5, 6), (16, 1, 4)])
def test_exact_arithmetic(N, g, K):
    """Gates in {1/2, 1, 2, -1}, values integers in [-4, 4], K <= 8: every
    product and every partial or total sum is k/2 with |k| <= 128, exact in
    fp32 and in bf16 (8 significant bits), so each partial is the exact sum
    over the slots on its node and y the exact sum over all slots, in any
    order."""
    rng = np.random.default_rng(N * 100 + g * 10 + K)
    T, d = 50, 16
    G = N * g
    a = rng.integers(0, G, size=(T, K)).astype(np.int32)
    pos = rng.permutation(T * K).reshape(T, K).astype(np.int32)
    vals = rng.integers(-4, 5, size=(T * K, d))
    eo = _bf16(vals.astype(np.float32))
    gates = rng.choice([0.5, 1.0, 2.0, -1.0], size=(T, K)).astype(np.float32)
    node_pos = _layout(a, N, g)
    part, y = oracle.node_combine(eo, pos, a, gates, node_pos, g)
    g64 = gates.astype(np.float64)
    v = vals.astype(np.float64)[pos]                       # [T, K, d]
    for t in range(T):
        for n in range(N):
            on = a[t] // g == n
            if node_pos[t, n] < 0:
                assert not on.any()
                continue
            want = (g64[t, on, None] * v[t, on]).sum(0)
            assert np.array_equal(_widen(part[node_pos[t, n]]), want)
    assert np.array_equal(_widen(y), (g64[:, :, None] * v).sum(1))


def test_partials_are_rounded_to_bf16_before_the_source_sum():
    """Worked by hand. Slot 0 on node 0: gate 1 + 2^-8 times 1. The product
    1 + 2^-8 lies halfway between the bf16 neighbours 1 and 1 + 2^-7, and
    rounding to even gives a partial of exactly 1. Slot 1 on node 1: gate 2^-8
    times 1, so its partial is 2^-8 exactly. The source sum 1 + 2^-8 ties
    again and rounds to 1. The plain combine adds in fp32 first:
    1 + 2^-8 + 2^-8 = 1 + 2^-7, which bf16 holds exactly."""
    a = np.array([[0, 1]], np.int32)                       # N = 2, g = 1
    pos = np.array([[0, 1]], np.int32)
    eo = _bf16([[1.0], [1.0]])
    gates = np.array([[1.0 + 2.0**-8, 2.0**-8]], np.float32)
    node_pos = _layout(a, 2, 1)
    part, y = oracle.node_combine(eo, pos, a, gates, node_pos, 1)
    assert _widen(part[node_pos[0, 0]])[0] == 1.0
    assert _widen(part[node_pos[0, 1]])[0] == 2.0**-8
    assert _widen(y)[0, 0] == 1.0
    flat, _ = oracle.combine(eo, pos, gates)
    assert _widen(flat)[0, 0] == 1.0 + 2.0**-7


def test_source_sums_in_increasing_node_order():
    """Worked by hand. Unit gates and one slot per node, with the slots in
    another order than the nodes: slot 0 holds -2^24 on node 2, slot 1 holds
    2^24 on node 0, slot 2 holds 1 on node 1. In increasing node order
    2^24 + 1 rounds back to 2^24 (a tie, to even), and adding -2^24 gives 0.
    The plain combine adds in slot order, -2^24 + 2^24 + 1, and gives 1."""
    a = np.array([[2, 0, 1]], np.int32)                    # N = 3, g = 1
    pos = np.array([[0, 1, 2]], np.int32)
    eo = _bf16([[-(2.0**24)], [2.0**24], [1.0]])
    gates = np.ones((1, 3), np.float32)
    node_pos = _layout(a, 3, 1)
    _, y = oracle.node_combine(eo, pos, a, gates, node_pos, 1)
    assert _widen(y)[0, 0] == 0.0
    flat, _ = oracle.combine(eo, pos, gates)
    assert _widen(flat)[0, 0] == 1.0


def test_skip_rules():
    """A slot with a rank outside [0, G) or a row outside [0, rows) adds
    nothing; a node row outside [0, node_rows) is neither written nor
    summed; a named node row with no slot of its token on the node holds
    zero."""
    N, g = 2, 2
    eo = _bf16([[1.0], [2.0], [4.0], [8.0]])
    gates = np.ones((1, 4), np.float32)
    a = np.array([[0, 3, -1, 1]], np.int32)
    pos = np.array([[0, 1, 2, 7]], np.int32)               # row 7 is out of range
    node_pos = np.array([[0, 1]], np.int32)
    part, y = oracle.node_combine(eo, pos, a, gates, node_pos, g)
    assert list(_widen(part)[:, 0]) == [1.0, 2.0]          # slots 2 and 3 skipped
    assert _widen(y)[0, 0] == 3.0
    # node 1's row beyond node_rows: not written, not summed
    part, y = oracle.node_combine(eo, pos, a, gates, np.array([[0, 5]], np.int32), g, node_rows=2)
    assert list(_widen(part)[:, 0]) == [1.0, 0.0]
    assert _widen(y)[0, 0] == 1.0
    # a named row for node 1 while no slot goes there: zero
    a2 = np.array([[0, 1, 0, 1]], np.int32)
    part, y = oracle.node_combine(eo, np.array([[0, 1, 2, 3]], np.int32), a2, gates, node_pos, g)
    assert list(_widen(part)[:, 0]) == [15.0, 0.0] and _widen(y)[0, 0] == 15.0


@pytest.mark.parametrize("name", ["clusters-e64", "colocate-e256", "drift-e384"])
def test_error_bound_against_the_plain_combine(name):
    """On a workload's routing, y differs from the plain combine by at most
    the roundings in between: each partial and both results round to bf16
    (unit roundoff 2^-8 each, at most 3 * 2^-8 of the sum of |g v| in all),
    plus the fp32 chains (2^-22 of it)."""
    w = W.with_sizes(W.WORKLOADS[name], T=W.WORKLOADS[name].G * 4, d=64)
    table, owner = W.layout(w, w.seed)
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    topk, gates = W.routing(w, w.seed)
    src = W.ragged_src(w.T, w.G, seed=1)
    a, _ = oracle.assign(w.N, w.g, w.E, tabs, topk.numpy(), src, seed=w.seed)
    _, _, pos, _ = oracle.dispatch(a, w.G, src)
    node_pos = oracle.node_dispatch(a, w.N, w.g, src=src)[2]
    eo = _bits(torch.randn(w.T * w.K, w.d).to(torch.bfloat16))
    gates = gates.numpy()
    part, y = oracle.node_combine(eo, pos, a, gates, node_pos, w.g)
    flat, _ = oracle.combine(eo, pos, gates)
    mag = np.abs(gates.astype(np.float64)[:, :, None] * _widen(eo)[pos]).sum(1)
    assert np.all(np.abs(_widen(y) - _widen(flat)) <= (3 * 2.0**-8 + 2.0**-22) * mag)
    # only the rows the layout names are written, and every one of them is
    named = np.zeros(len(part), bool)
    named[node_pos[node_pos >= 0]] = True
    assert named.all()
