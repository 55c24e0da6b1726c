"""Both combines on expert outputs that hold special bf16 values, against
the oracle bit for bit: infinities, sums that overflow fp32 to infinity,
denormal inputs and results, signed zeros, and sums that sit on a bf16
rounding tie. The kernels round with the hardware's packed bf16
conversion, the oracle with the IEEE-754 rule written out, so these cases
pin the two against each other where the rule has its special branches.
NaN inputs and sums of opposite infinities are left out: which NaN an fp32
operation returns from such operands is not fixed by IEEE-754 and differs
between the GPU and the host."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import pipeline as PL
from paper_2609_36959_amd import workload as W

pytestmark = pytest.mark.gpu

SENTINEL = 0x7FA5  # a NaN pattern no output row can hold


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    B.lib()
    yield
    torch.cuda.synchronize()


def dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a, dtype)).cuda()


def bf16_dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits, np.uint16).view(np.int16)).view(
        torch.bfloat16).cuda()


def special_inputs(w, seed):
    """The oracle's routing for w, and expert rows and gates with special
    values in chosen columns. Column classes (d = 1032, a ragged last slice):
    +inf in some rows; -inf in some rows (other columns); the largest finite
    bf16 everywhere (overflow where a token's gates sum above 1); bf16
    denormals; signed zeros; small exact values whose sums land on ties."""
    table, owner = W.layout(w, seed)
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    topk, _ = W.routing(w, seed)
    src = W.ragged_src(w.T, w.G, seed=seed)
    a, _ = oracle.assign(w.N, w.g, w.E, tabs, topk.numpy(), src, seed=seed)
    _, _, pos, _ = oracle.dispatch(a, w.G, src)
    node_pos = oracle.node_dispatch(a, w.N, w.g, src=src)[2]
    rng = np.random.default_rng(seed)
    rows, d = w.T * w.K, w.d
    gen = torch.Generator().manual_seed(seed)
    eo = PL.bf16_bits(torch.randn(rows, d, generator=gen).to(torch.bfloat16)).copy()
    col = rng.permutation(d)
    pinf, ninf, big, den, zer, tie = np.split(col[:6 * 64], 6)
    some = rng.random(rows) < 0.2
    eo[np.ix_(some, pinf)] = 0x7F80
    eo[np.ix_(rng.random(rows) < 0.2, ninf)] = 0xFF80
    eo[:, big] = 0x7F7F
    eo[:, den] = rng.integers(1, 0x80, size=(rows, den.size)) | (
        rng.integers(0, 2, size=(rows, den.size)) << 15)
    eo[:, zer] = rng.choice([0x0000, 0x8000], size=(rows, zer.size))
    # exact multiples of 2^-8 in [1, 2): with gate 1 the sums often need one
    # bit more than bf16 keeps, and then sit on a tie
    eo[:, tie] = 0x3F80 + rng.integers(0, 0x80, size=(rows, tie.size))
    gates = rng.random((w.T, w.K)).astype(np.float32) + np.float32(0.01)
    gates[rng.random(w.T) < 0.3] = 1.0   # K times the largest value overflows
    gates[rng.random(w.T) < 0.1] = 2.0
    denorm_gate = rng.random(w.T) < 0.2  # products below the normal range
    gates[denorm_gate] = np.float32(2.0 ** -100)
    return a, pos, node_pos, eo.astype(np.uint16), gates


@pytest.mark.parametrize("name", ["clusters-e64", "colocate-e128"])
def test_special_values(name):
    w = W.with_sizes(W.WORKLOADS[name], T=W.WORKLOADS[name].G * 3 + 11, d=1032)
    a, pos, node_pos, eo, gates = special_inputs(w, w.seed)
    print(f"special values {name} T={w.T} d={w.d}", flush=True)
    ref_y, _ = oracle.combine(eo, pos, gates)
    # the cases are there: infinities, finite maxima, denormal and tie results
    assert np.any(ref_y == 0x7F80) and np.any(ref_y == 0xFF80)
    assert np.any(((ref_y & 0x7F80) == 0) & ((ref_y & 0x7F) != 0))
    assert np.any(ref_y == 0x8000)
    y = torch.full((w.T, w.d), SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    B.cobalt_combine(bf16_dev(eo), dev(pos, np.int32), dev(gates, np.float32), y)
    torch.cuda.synchronize()
    assert np.array_equal(PL.bf16_bits(y), ref_y)

    cap = w.T * min(w.K, w.N)
    ref_part, ref_ny = oracle.node_combine(eo, pos, a, gates, node_pos, w.g, node_rows=cap)
    part = torch.full((cap, w.d), SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    ny = torch.full((w.T, w.d), SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    B.cobalt_node_combine(bf16_dev(eo), dev(pos, np.int32), dev(a, np.int32),
                          dev(gates, np.float32), dev(node_pos, np.int32), w.N, w.g, part, ny)
    torch.cuda.synchronize()
    named = np.zeros(cap, bool)
    named[node_pos[(node_pos >= 0) & (node_pos < cap)]] = True
    assert np.array_equal(PL.bf16_bits(part)[named], ref_part[named])
    assert np.array_equal(PL.bf16_bits(ny), ref_ny)
