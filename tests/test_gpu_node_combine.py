"""GPU parity of the node-level combine (per-node bf16 partials, then the
source-side sum in node order), called through the C ABI, against the
oracle bit for bit: every named partial row and every row of y; rows the
layout does not name keep their contents. Routing inputs (assignment, pos,
node_pos) come from the oracle. Sizes span several slices and ragged token
counts; edge cases cover one node, 16 nodes, K = 1, K = 16, 16-byte rows,
rows wider than the 16 slices of the templated kernels, skipped slots and
node rows, and empty inputs. The full-size case runs the benchmark's
workload and checks sampled tokens."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import pipeline as PL
from paper_2609_36959_amd import workload as W

pytestmark = pytest.mark.gpu

SENTINEL = 0x7FA5  # a NaN pattern no partial row can hold


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    B.lib()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a, dtype)).cuda()


def bf16_dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def run(eo_bits, pos, assigned, gates, node_pos, N, g):
    T, K = pos.shape
    d = eo_bits.shape[1]
    cap = T * min(K, N)
    partial = torch.full((cap, d), SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    y = torch.full((T, d), SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    B.cobalt_node_combine(bf16_dev(eo_bits), dev(pos, np.int32), dev(assigned, np.int32),
                          dev(gates, np.float32), dev(node_pos, np.int32), N, g, partial, y)
    torch.cuda.synchronize()
    return PL.bf16_bits(partial), PL.bf16_bits(y)


def check(eo_bits, pos, assigned, gates, node_pos, N, g):
    T, K = pos.shape
    cap = T * min(K, N)
    ref_part, ref_y = oracle.node_combine(eo_bits, pos, assigned, gates, node_pos, g,
                                          node_rows=cap)
    got_part, got_y = run(eo_bits, pos, assigned, gates, node_pos, N, g)
    assert np.array_equal(got_y, ref_y), "y differs"
    named = np.zeros(cap, bool)
    q = node_pos[(node_pos >= 0) & (node_pos < cap)]
    named[q] = True
    assert np.array_equal(got_part[named], ref_part[named]), "partial rows differ"
    assert np.all(got_part[~named] == SENTINEL), "a row the layout does not name was written"


def routed(w, seed, src_kind="ragged"):
    """The oracle's assignment, per-pair rows and node rows for w."""
    table, owner = W.layout(w, seed)
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    topk, gates = W.routing(w, seed)
    src = W.ragged_src(w.T, w.G, seed=seed) if src_kind == "ragged" else None
    a, _ = oracle.assign(w.N, w.g, w.E, tabs, topk.numpy(), src, seed=seed)
    _, _, pos, _ = oracle.dispatch(a, w.G, src)
    node_pos = oracle.node_dispatch(a, w.N, w.g, src=src)[2]
    return a, pos, node_pos, gates.numpy()


def eo_for(rows, d, seed):
    gen = torch.Generator().manual_seed(seed)
    return PL.bf16_bits(torch.randn(rows, d, generator=gen).to(torch.bfloat16))


@pytest.mark.parametrize("name", W.NAMES)
@pytest.mark.parametrize("d", [256, 7168])
def test_workloads(name, d):
    base = W.WORKLOADS[name]
    T = base.G * 6 + 37 if d == 256 else base.G * 2 + 5
    w = W.with_sizes(base, T=T, d=d)
    print(f"node combine {name} T={T} d={d}", flush=True)
    a, pos, node_pos, gates = routed(w, w.seed)
    check(eo_for(w.T * w.K, d, w.seed), pos, a, gates, node_pos, w.N, w.g)


@pytest.mark.parametrize("N,g,K,d", [(1, 8, 8, 64), (16, 1, 16, 64), (4, 2, 1, 64),
                                     (8, 8, 8, 8), (4, 2, 8, 16392), (2, 4, 3, 1032)])
def test_edge_shapes(N, g, K, d):
    """One node (y equals the plain combine), 16 nodes with K = 16, K = 1,
    16-byte rows, rows of 17 slices (the kernels' run-time slice count), and
    a ragged last slice."""
    rng = np.random.default_rng(N * 1000 + K * 10 + d)
    G = N * g
    T = 3 * G + 11 if d < 8192 else 2 * G + 3
    print(f"node combine edge N={N} g={g} K={K} d={d} T={T}", flush=True)
    a = np.stack([rng.choice(G, size=K, replace=K > G) for _ in range(T)]).astype(np.int32)
    src = np.sort(rng.integers(0, G, size=T)).astype(np.int32)
    _, _, pos, _ = oracle.dispatch(a, G, src)
    node_pos = oracle.node_dispatch(a, N, g, src=src)[2]
    gates = rng.random((T, K)).astype(np.float32)
    eo = eo_for(T * K, d, int(rng.integers(1 << 30)))
    check(eo, pos, a, gates, node_pos, N, g)
    if N == 1:
        flat, _ = oracle.combine(eo, pos, gates)
        _, got_y = run(eo, pos, a, gates, node_pos, N, g)
        assert np.array_equal(got_y, flat)


def test_skipped_slots_and_node_rows():
    """Slots with a rank outside [0, G) or a row outside [0, T*K) add
    nothing; node_pos entries outside [0, T*min(K, N)) are neither written
    nor summed; a named row for a node no slot of the token reaches holds
    zero."""
    rng = np.random.default_rng(5)
    N, g, K, d = 4, 2, 6, 136
    G = N * g
    T = 200
    a = rng.integers(0, G, size=(T, K)).astype(np.int32)
    src = np.sort(rng.integers(0, G, size=T)).astype(np.int32)
    _, _, pos, _ = oracle.dispatch(a, G, src)
    node_pos = oracle.node_dispatch(a, N, g, src=src)[2]
    cap = T * min(K, N)
    bad = rng.random((T, K))
    a2, pos2, np2 = a.copy(), pos.copy(), node_pos.copy()
    a2[bad < 0.05] = -1
    a2[(bad >= 0.05) & (bad < 0.08)] = G + 3
    pos2[(bad >= 0.08) & (bad < 0.12)] = -5
    pos2[(bad >= 0.12) & (bad < 0.15)] = T * K + 9
    sel = rng.random((T, N)) < 0.05
    np2[sel & (np2 >= 0)] = cap + 7                    # named beyond the buffer: skipped
    extra = (np2 < 0) & (rng.random((T, N)) < 0.01)    # named, but no slot on the node
    unused = np.setdiff1d(np.arange(cap), np2[np2 >= 0])
    np2[extra] = unused[:int(extra.sum())]
    gates = rng.standard_normal((T, K)).astype(np.float32)
    check(eo_for(T * K, d, 9), pos2, a2, gates, np2, N, g)


def test_empty_input():
    N, g, K, d = 2, 2, 4, 64
    partial = torch.zeros(0, d, dtype=torch.bfloat16, device="cuda")
    y = torch.zeros(0, d, dtype=torch.bfloat16, device="cuda")
    z = torch.zeros(0, K, dtype=torch.int32, device="cuda")
    B.cobalt_node_combine(torch.zeros(0, d, dtype=torch.bfloat16, device="cuda"), z, z,
                          torch.zeros(0, K, device="cuda"),
                          torch.zeros(0, N, dtype=torch.int32, device="cuda"), N, g, partial, y)
    torch.cuda.synchronize()


def test_full_size_sampled_tokens():
    """colocate-e256 at full size (T=131072, K=8, d=7168): the step's own
    assignment, rows and node rows (checked against the oracle's), then the
    node-level combine on the step's expert outputs; 256 seeded tokens are
    checked against the oracle, which takes just their rows."""
    w = W.WORKLOADS["colocate-e256"]
    print(f"node combine full size {w.describe()}", flush=True)
    st = PL.RoutingStep(w, seed=w.seed, device="cuda")
    st.run()
    st.node_pack()
    torch.cuda.synchronize()
    tabs = oracle.layout_tables(w.N, w.g, w.E, st.table, st.owner)
    a, _ = oracle.assign(w.N, w.g, w.E, tabs, st.topk.cpu().numpy(), None, seed=st.seed,
                         step=st.step)
    _, _, pos, _ = oracle.dispatch(a, w.G)
    node_pos = oracle.node_dispatch(a, w.N, w.g)[2]
    assert np.array_equal(st.assigned.cpu().numpy(), a)
    assert np.array_equal(st.pos.cpu().numpy(), pos)
    assert np.array_equal(st.node_pos.cpu().numpy(), node_pos)
    cap = w.T * min(w.K, w.N)
    partial = torch.empty(cap, w.d, dtype=torch.bfloat16, device="cuda")
    y = torch.empty(w.T, w.d, dtype=torch.bfloat16, device="cuda")
    B.cobalt_node_combine(st.eo, st.pos, st.assigned, st.gates, st.node_pos, w.N, w.g, partial, y)
    torch.cuda.synchronize()
    rng = np.random.default_rng(w.seed)
    t = np.sort(rng.choice(w.T, size=256, replace=False))
    eo_rows = PL.bf16_bits(st.eo[torch.from_numpy(pos[t].ravel().astype(np.int64)).cuda()])
    ident = np.arange(len(t) * w.K, dtype=np.int32).reshape(len(t), w.K)
    np_t = node_pos[t]
    renum = np.full_like(np_t, -1)
    renum[np_t >= 0] = np.arange(int((np_t >= 0).sum()), dtype=np.int32)
    ref_part, ref_y = oracle.node_combine(eo_rows, ident, a[t], st.gates.cpu().numpy()[t], renum,
                                          w.g)
    got_rows = PL.bf16_bits(partial[torch.from_numpy(np_t[np_t >= 0].astype(np.int64)).cuda()])
    assert np.array_equal(got_rows, ref_part[renum[np_t >= 0]])
    assert np.array_equal(PL.bf16_bits(y[torch.from_numpy(t).cuda()]), ref_y)
    st.close()
    del st, partial, y
    torch.cuda.empty_cache()
