"""GPU parity of the node-deduplicated dispatch layout and pack, called
through the C ABI, against the oracle element by element: node counts,
offsets, node_pos, forwarding masks, row tokens and packed rows, all bit
exact. Sizes span several look-back tiles with ragged tails; edge cases
cover one node, 16 nodes, one rank per node, K = 1 and K = 16, tiny and long
rows, empty inputs, index-only calls and skipped out-of-range ranks. The
full-size case runs the benchmark's workload in its launch configuration."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import pipeline as PL
from paper_2609_36959_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    B.lib()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def dev_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()


def run_node(assigned, src, N, g, x_bits, repeat=1, with_tokens=True):
    """Runs cobalt_node_dispatch_pack; returns host copies of each repeat's
    outputs, trimmed to the rows used."""
    T, K = assigned.shape
    G, cap = N * g, T * min(K, N)
    t_a = dev_i32(assigned)
    t_src = None if src is None else dev_i32(src)
    x = None
    if x_bits is not None:
        x = torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).view(torch.bfloat16).cuda()
    counts = torch.full((G, N), -1, dtype=torch.int32, device="cuda")
    offsets = torch.full((G * N + 1,), -1, dtype=torch.int64, device="cuda")
    node_pos = torch.full((T, N), -9, dtype=torch.int32, device="cuda")
    fwd = torch.full((cap,), -9, dtype=torch.int32, device="cuda")
    tok = torch.full((cap,), -9, dtype=torch.int32, device="cuda") if with_tokens else None
    packed = None if x is None else torch.zeros(cap, x.shape[1], dtype=torch.bfloat16,
                                                device="cuda")
    ws = B.node_workspace_for(T, N, g)
    ws.fill_(0xCD)  # contents on entry must not matter
    outs = []
    for _ in range(repeat):
        B.cobalt_node_dispatch_pack(t_a, t_src, N, g, x, counts, offsets, node_pos, fwd, tok,
                                    packed, ws)
        torch.cuda.synchronize()
        o = offsets.cpu().numpy()
        rows = int(o[-1])
        outs.append(dict(counts=counts.cpu().numpy(), offsets=o, node_pos=node_pos.cpu().numpy(),
                         fwd=fwd.cpu().numpy().view(np.uint32)[:rows],
                         tok=None if tok is None else tok.cpu().numpy()[:rows],
                         packed=None if packed is None else PL.bf16_bits(packed)[:rows]))
    return outs


def check(assigned, src, N, g, d, seed, repeat=1, ref_assigned=None):
    T = assigned.shape[0]
    x_bits = None
    if d:
        gen = torch.Generator().manual_seed(seed)
        x_bits = PL.bf16_bits(torch.randn(T, d, generator=gen).to(torch.bfloat16))
    ref = oracle.node_dispatch(assigned if ref_assigned is None else ref_assigned, N, g, src,
                               x_bits)
    for got in run_node(assigned, src, N, g, x_bits, repeat):
        assert np.array_equal(got["counts"], ref[0])
        assert np.array_equal(got["offsets"], ref[1])
        assert np.array_equal(got["node_pos"], ref[2])
        assert np.array_equal(got["fwd"], ref[3])
        assert np.array_equal(got["tok"], ref[4])
        if d:
            assert np.array_equal(got["packed"], ref[5])
    return ref


CASES = [
    # workload, T, d, source ranks
    ("tiny", 4096, 512, "null"),
    ("tiny", 3001, 128, "ragged"),
    ("clusters-e64", 5003, 256, "ragged"),
    ("colocate-e128", 32 * 130, 1024, "null"),
    ("colocate-e256", 64 * 40 + 64 * 9, 7168, "null"),
    ("colocate-e256", 2999, 64, "ragged"),
    ("drift-e384", 64 * 333, 256, "null"),
]


@pytest.mark.parametrize("name,T,d,srckind", CASES)
@pytest.mark.parametrize("mode", [0, 1])
def test_node_layout_matches_oracle(name, T, d, srckind, mode):
    w = W.with_sizes(W.WORKLOADS[name], T=T, d=d)
    print(f"node case {name} T={T} d={d} src={srckind} mode={mode}", flush=True)
    topk, _ = W.routing(w, w.seed)
    table, owner = W.layout(w, w.seed)
    src = None if srckind == "null" else W.ragged_src(T, w.G, seed=w.seed)
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    a, rn = oracle.assign(w.N, w.g, w.E, tabs, topk.numpy(), src, seed=w.seed, step=2, mode=mode)
    ref = check(a, src, w.N, w.g, d, seed=T)
    s = W.contiguous_src(T, w.G) if src is None else src
    home = s // w.g
    cross = int((ref[2] >= 0).sum()) - int((ref[2][np.arange(T), home] >= 0).sum())
    assert cross == oracle.traffic(a, w.N, w.g, src)[0]  # Eq. 1's V


@pytest.mark.parametrize("N,g,T,K,d", [
    (1, 4, 4 * 301, 3, 64),       # one node: every row is local
    (16, 2, 32 * 41, 8, 32),      # 16 nodes (generic copy path)
    (4, 8, 32 * 50, 1, 8),        # K = 1 and one-vector rows
    (2, 4, 8 * 90, 16, 8200),     # K = 16 > N; rows of 1025 vectors
    (8, 1, 8 * 700, 4, 16),       # one rank per node
    (16, 32, 512 * 3, 8, 16),     # G = 512, largest bucket matrix
])
def test_edge_shapes(N, g, T, K, d):
    rng = np.random.default_rng(N * 1000 + g * 10 + K)
    a = rng.integers(0, N * g, size=(T, K)).astype(np.int32)
    check(a, None, N, g, d, seed=K)
    check(a, W.ragged_src(T, N * g, seed=3), N, g, d, seed=K)


def test_repeats_are_identical_with_a_stale_workspace():
    rng = np.random.default_rng(8)
    a = rng.integers(0, 64, size=(512 * 9 + 13, 8)).astype(np.int32)
    check(a, W.ragged_src(a.shape[0], 64, seed=4), 8, 8, 64, seed=1, repeat=3)


def test_out_of_range_ranks_are_skipped():
    """A slot whose rank is outside [0, G) adds no row and no mask bit: the
    result equals the oracle's on the data where that slot repeats another
    slot of the same token."""
    rng = np.random.default_rng(12)
    N, g, T, K = 4, 4, 16 * 129, 4
    a = rng.integers(0, N * g, size=(T, K)).astype(np.int32)
    ref_a = a.copy()
    bad = rng.choice(T, size=200, replace=False)
    a[bad, 0] = np.where(np.arange(200) % 2 == 0, -1, N * g + 3)
    ref_a[bad, 0] = ref_a[bad, 1]
    check(a, None, N, g, 32, seed=2, ref_assigned=ref_a)


def test_index_only_and_empty():
    rng = np.random.default_rng(3)
    a = rng.integers(0, 32, size=(32 * 77, 6)).astype(np.int32)
    ref = oracle.node_dispatch(a, 4, 8)
    got = run_node(a, None, 4, 8, None, with_tokens=False)[0]
    assert np.array_equal(got["node_pos"], ref[2]) and np.array_equal(got["fwd"], ref[3])
    got = run_node(np.zeros((0, 4), np.int32), np.zeros(0, np.int32), 2, 2, None)[0]
    assert not got["counts"].any() and not got["offsets"].any()


def test_full_size_node_pack():
    """The benchmark's workload (T=131072, E=256, K=8, d=7168, 8x8 ranks) in
    its launch configuration: the layout is compared in full with the
    oracle, packed rows on a seeded sample."""
    w = W.WORKLOADS["colocate-e256"]
    print(f"full size node pack {w.describe()}", flush=True)
    st = PL.RoutingStep(w, seed=w.seed, device="cuda")
    st.assign()
    st.node_pack()
    torch.cuda.synchronize()
    a = st.assigned.cpu().numpy()
    counts, offsets, node_pos, fwd, tok, _ = oracle.node_dispatch(a, w.N, w.g)
    rows = int(offsets[-1])
    assert np.array_equal(st.node_counts.cpu().numpy(), counts)
    assert np.array_equal(st.node_offsets.cpu().numpy(), offsets)
    assert np.array_equal(st.node_pos.cpu().numpy(), node_pos)
    assert np.array_equal(st.fwd_mask.cpu().numpy().view(np.uint32)[:rows], fwd)
    assert np.array_equal(st.row_token.cpu().numpy()[:rows], tok)
    rng = np.random.default_rng(7)
    r = np.sort(rng.choice(rows, size=4096, replace=False))
    got = PL.bf16_bits(st.node_packed[torch.from_numpy(r).cuda()])
    want = PL.bf16_bits(st.x[torch.from_numpy(tok[r].astype(np.int64)).cuda()])
    assert np.array_equal(got, want)
    V = oracle.traffic(a, w.N, w.g)[0]
    home = W.contiguous_src(w.T, w.G) // w.g
    assert rows - int((node_pos[np.arange(w.T), home] >= 0).sum()) == V
    st.close()
    del st
    torch.cuda.empty_cache()
