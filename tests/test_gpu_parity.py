"""GPU parity: every step of the HIP path, called through the C ABI, against
the oracle on the same seeded inputs, element by element. Sizes span
several tiles with ragged tails; edge cases cover empty inputs, K = 1, one
node, 16 nodes, tiny and long rows, and the row bands of the statistics
histogram."""
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


def u32(t):
    return t.cpu().numpy().view(np.uint32)


def dev_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()


def bits_to_bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.uint16).view(np.int16)).view(torch.bfloat16).cuda()


def run_path(w, seed, topk, gates, table, owner, src=None, x_bits=None, eo_bits=None, step=0,
             mode=0, repeat=1):
    """Runs the four calls on the GPU; returns host copies of every output."""
    T, K, E, G, d = topk.shape[0], w.K, w.E, w.G, w.d
    L = B.cobalt_layout_create(w.N, w.g, E, table.shape[1], table, owner)
    t_topk = dev_i32(topk)
    t_src = None if src is None else dev_i32(src)
    coact = torch.zeros(E, E, dtype=torch.int32, device="cuda")
    count = torch.zeros(E, dtype=torch.int32, device="cuda")
    B.cobalt_coact_stats(t_topk, E, coact, count, B.stats_workspace_for(T, K, E))
    assigned = torch.full((T, K), -7, dtype=torch.int32, device="cuda")
    remote = torch.zeros(T, dtype=torch.int16, device="cuda")
    B.cobalt_assign(L, t_topk, t_src, seed, step, mode, assigned, remote)
    x = bits_to_bf16(x_bits)
    counts = torch.full((G, G), -1, dtype=torch.int32, device="cuda")
    offsets = torch.full((G * G + 1,), -1, dtype=torch.int64, device="cuda")
    pos = torch.full((T, K), -1, dtype=torch.int32, device="cuda")
    packed = torch.zeros(T * K, d, dtype=torch.bfloat16, device="cuda")
    ws = B.workspace_for(T, K, G)
    ws.fill_(0xAB)  # contents on entry must not matter
    outs = []
    for _ in range(repeat):
        B.cobalt_dispatch_pack(assigned, t_src, G, x, counts, offsets, pos, packed, ws)
        outs.append((counts.cpu().numpy(), offsets.cpu().numpy(), pos.cpu().numpy(),
                     PL.bf16_bits(packed)))
    eo = bits_to_bf16(eo_bits)
    y = torch.zeros(T, d, dtype=torch.bfloat16, device="cuda")
    y32 = torch.zeros(T, d, dtype=torch.float32, device="cuda")
    B.cobalt_combine(eo, pos, dev_gates(gates), y, y32)
    torch.cuda.synchronize()
    res = dict(coact=u32(coact), count=u32(count), assigned=assigned.cpu().numpy(),
               remote=remote.cpu().numpy().view(np.uint16), dispatch=outs,
               y=PL.bf16_bits(y), y32=y32.cpu().numpy(), tables=B.cobalt_layout_tables(L))
    B.cobalt_layout_destroy(L)
    return res


def dev_gates(g):
    return torch.from_numpy(np.ascontiguousarray(g, np.float32)).cuda()


def check_against_oracle(w, seed, topk, gates, table, owner, src=None, step=0, mode=0, repeat=1):
    T, K, E, G, d = topk.shape[0], w.K, w.E, w.G, w.d
    gen = torch.Generator().manual_seed(seed + 17)
    x_bits = PL.bf16_bits(torch.randn(T, d, generator=gen).to(torch.bfloat16))
    eo_bits = PL.bf16_bits(torch.randn(T * K, d, generator=gen).to(torch.bfloat16))
    got = run_path(w, seed, topk, gates, table, owner, src, x_bits, eo_bits, step, mode, repeat)

    tabs = oracle.layout_tables(w.N, w.g, E, table, owner)
    for mine, ref in zip(got["tables"], tabs):
        assert np.array_equal(mine.view(ref.dtype), ref)
    C, cnt = oracle.coact_stats(topk, E)
    assert np.array_equal(got["coact"], C)
    assert np.array_equal(got["count"], cnt)
    a, rn = oracle.assign(w.N, w.g, E, tabs, topk, src, seed=seed, step=step, mode=mode)
    assert np.array_equal(got["assigned"], a)
    assert np.array_equal(got["remote"], rn)
    counts, offsets, pos, packed = oracle.dispatch(a, G, src, x_bits)
    for c2, o2, p2, pk2 in got["dispatch"]:
        assert np.array_equal(c2, counts)
        assert np.array_equal(o2, offsets)
        assert np.array_equal(p2, pos)
        assert np.array_equal(pk2, packed)
    y, y32 = oracle.combine(eo_bits, pos, gates)
    # acceptance bar: fp32 sums within 1e-3 of the oracle's, relative to the
    # magnitude of the terms; the kernel keeps the oracle's order, so the
    # results are in fact identical bit for bit
    v = torch.from_numpy(eo_bits.view(np.int16)).view(torch.bfloat16).double().numpy()[pos]
    scale = (np.abs(gates.astype(np.float64))[:, :, None] * np.abs(v)).sum(1)
    assert np.all(np.abs(got["y32"].astype(np.float64) - y32) <= 1e-3 * scale + 1e-30)
    assert np.array_equal(got["y32"].view(np.uint32), y32.view(np.uint32))
    assert np.array_equal(got["y"], y)
    return got


CASES = [
    # workload, T, d, source ranks
    ("tiny", 4096, 512, "null"),
    ("tiny", 4096 + 8 * 37, 512, "null"),
    ("tiny", 3001, 128, "ragged"),
    ("clusters-e64", 32 * 200, 2048, "null"),
    ("clusters-e64", 5003, 256, "ragged"),
    ("colocate-e128", 32 * 130, 4096, "null"),
    ("colocate-e256", 64 * 40, 7168, "null"),
    ("colocate-e256", 2999, 64, "ragged"),
    ("drift-e384", 64 * 33, 1024, "null"),
]


@pytest.mark.parametrize("name,T,d,srckind", CASES)
@pytest.mark.parametrize("mode", [0, 1])
def test_path_matches_oracle(name, T, d, srckind, mode):
    w = W.with_sizes(W.WORKLOADS[name], T=T, d=d)
    print(f"case {name} T={T} d={d} src={srckind} mode={mode}", flush=True)
    topk, gates = W.routing(w, w.seed)
    table, owner = W.layout(w, w.seed)
    src = None if srckind == "null" else W.ragged_src(T, w.G, seed=w.seed)
    check_against_oracle(w, w.seed, topk.numpy(), gates.numpy(), table, owner, src, step=3,
                         mode=mode)


def test_deterministic_repeats_and_stale_workspace():
    w = W.with_sizes(W.WORKLOADS["colocate-e256"], T=64 * 70, d=256)
    topk, gates = W.routing(w, 5)
    table, owner = W.layout(w, 5)
    got = check_against_oracle(w, 5, topk.numpy(), gates.numpy(), table, owner, repeat=4)
    first = got["dispatch"][0]
    for other in got["dispatch"][1:]:
        for a, b in zip(first, other):
            assert np.array_equal(a, b)


def test_statistics_accumulate_across_calls():
    w = W.with_sizes(W.WORKLOADS["drift-e384"], T=64 * 40)
    E = w.E
    coact = torch.zeros(E, E, dtype=torch.int32, device="cuda")
    count = torch.zeros(E, dtype=torch.int32, device="cuda")
    C = np.zeros((E, E), np.uint32)
    cnt = np.zeros(E, np.uint32)
    for step in range(3):
        topk, _ = W.routing(w, 4, step=step)
        B.cobalt_coact_stats(topk.cuda(), E, coact, count, B.stats_workspace_for(w.T, w.K, E))
        C, cnt = oracle.coact_stats(topk.numpy(), E, C, cnt)
    torch.cuda.synchronize()
    assert np.array_equal(u32(coact), C) and np.array_equal(u32(count), cnt)


@pytest.mark.parametrize("E,T", [(384, 3000), (384, 70001), (1024, 3000), (4096, 2500),
                                 (2, 3000), (1, 100), (256, 131072 + 77)])
def test_statistics_layouts(E, T):
    """Pair histograms in LDS as one band (E = 1, 2; small calls), in the
    four interleaved row bands of large calls (E = 256, 384), and in as many
    bands as the LDS needs (E = 384 at small T: 2, E = 1024: 16, E = 4096:
    256), over one or many token chunks with ragged tails."""
    rng = np.random.default_rng(E + T)
    K = min(8, E)
    topk = np.argsort(rng.random((T, E)), axis=1)[:, :K].astype(np.int32)
    coact = torch.zeros(E, E, dtype=torch.int32, device="cuda")
    count = torch.zeros(E, dtype=torch.int32, device="cuda")
    B.cobalt_coact_stats(dev_i32(topk), E, coact, count, B.stats_workspace_for(T, K, E))
    C, cnt = oracle.coact_stats(topk, E)
    assert np.array_equal(u32(coact), C)
    assert np.array_equal(u32(count), cnt)


def _stats_check(topk, E):
    T, K = topk.shape
    coact = torch.zeros(E, E, dtype=torch.int32, device="cuda")
    count = torch.zeros(E, dtype=torch.int32, device="cuda")
    B.cobalt_coact_stats(dev_i32(topk), E, coact, count, B.stats_workspace_for(T, K, E))
    C, cnt = oracle.coact_stats(topk, E)
    assert np.array_equal(u32(coact), C)
    assert np.array_equal(u32(count), cnt)


def test_statistics_uint32_partials():
    """K = 16 over 140 000 tokens: 128 chunks of 1094 tokens could pass
    65535 in a bin (64 per token at most), so the partials are uint32."""
    rng = np.random.default_rng(11)
    T, E, K = 140000, 64, 16
    _stats_check(np.argsort(rng.random((T, E)), axis=1)[:, :K].astype(np.int32), E)


def test_statistics_uint16_bound():
    """128 chunks of 4095 tokens that each add 16 to the pair (3, 5) (ids 3
    and 5 four times each): every chunk's bin holds 65520, the most a uint16
    partial is trusted with."""
    T = 4095 * 128
    topk = np.tile(np.array([3, 3, 3, 3, 5, 5, 5, 5], np.int32), (T, 1))
    _stats_check(topk, 16)


def _stats_valid_slots(topk, E):
    """The statistics with ids outside [0, E) dropped: every ordered pair of
    distinct slots whose ids are both in range, and every such slot."""
    T, K = topk.shape
    C = np.zeros((E, E), np.uint64)
    cnt = np.zeros(E, np.uint64)
    ok = (topk >= 0) & (topk < E)
    for a in range(K):
        np.add.at(cnt, topk[ok[:, a], a], 1)
        for b in range(K):
            if a != b:
                m = ok[:, a] & ok[:, b]
                np.add.at(C, (topk[m, a], topk[m, b]), 1)
    return C.astype(np.uint32), cnt.astype(np.uint32)


@pytest.mark.parametrize("T,E", [(3 * 2048 + 5, 40), (131072 + 5, 256)])
def test_statistics_mixed_waves(T, E):
    """Tokens with repeated ids (m copies add m(m - 1) to the diagonal) or
    out-of-range ids (which count nowhere) scattered among valid ones, so
    that some waves take the per-pair checks and the rest skip them; the
    second size runs the two-band plan with uint16 partials."""
    rng = np.random.default_rng(12)
    K = 8
    topk = np.argsort(rng.random((T, E)), axis=1)[:, :K].astype(np.int32)
    rows = rng.choice(T, size=60, replace=False)
    topk[rows[:20], 3] = topk[rows[:20], 6]            # an id twice
    topk[rows[20:30], 1:4] = topk[rows[20:30], :1]     # an id four times
    topk[rows[30:], 0] = rng.choice([-1, E, -7], size=30)  # out of range
    # the brute force agrees with the oracle where every id is in range
    good = np.setdiff1d(np.arange(T), rows[30:])
    assert all(np.array_equal(x, y) for x, y in
               zip(_stats_valid_slots(topk[good], E), oracle.coact_stats(topk[good], E)))
    C, cnt = _stats_valid_slots(topk, E)
    coact = torch.zeros(E, E, dtype=torch.int32, device="cuda")
    count = torch.zeros(E, dtype=torch.int32, device="cuda")
    B.cobalt_coact_stats(dev_i32(topk), E, coact, count, B.stats_workspace_for(T, K, E))
    assert np.array_equal(u32(coact), C)
    assert np.array_equal(u32(count), cnt)


def _custom(N, g, E, S, K, T, d, seed, extra_per_rank=None):
    w = W.Workload("custom", T, E, K, d, N, g, S)
    rng = np.random.default_rng(seed)
    G = N * g
    per = E // G
    slots = [list(range(r * per, (r + 1) * per)) for r in range(G)]
    for e in rng.permutation(E):
        cand = [r for r in range(G) if len(slots[r]) < S and e not in slots[r]]
        if cand and rng.random() < 0.7:
            slots[cand[rng.integers(len(cand))]].append(int(e))
    table = np.full((G, S), -1, np.int32)
    for r in range(G):
        table[r, : len(slots[r])] = slots[r]
    owner = (np.arange(E) // per).astype(np.int32)
    topk = np.stack([rng.choice(E, size=K, replace=False) for _ in range(T)]).astype(np.int32)
    g_ = rng.random((T, K)).astype(np.float32)
    gates = (g_ / g_.sum(1, keepdims=True)).astype(np.float32)
    return w, topk, gates, table, owner


@pytest.mark.parametrize("N,g,E,S,K,T,d", [
    (1, 4, 16, 6, 3, 4 * 301, 64),      # one node: nothing remote
    (16, 2, 64, 4, 8, 32 * 41, 32),     # 16 nodes: 15-bit remote masks
    (4, 8, 64, 3, 1, 32 * 50, 8),       # K = 1 and one-vector rows
    (2, 4, 16, 4, 16, 8 * 90, 8200),    # K = 16; rows of 1025 vectors (long copy path)
    (8, 1, 8, 3, 4, 8 * 100, 16),       # one GPU per node
    (2, 4, 16, 4, 4, 8 * 16, 16392),    # 17 slices of 2 KiB: the fan-out pack and
                                        # one-wave-per-token combine
    (2, 4, 16, 4, 8, 8 * 16, 16384),    # 16 slices: the largest scatter / fold shape
    (16, 8, 1024, 12, 8, 128 * 24, 64),  # E = 1024, G = 128: row-band statistics
    (16, 32, 4096, 12, 8, 512 * 6, 16),  # E = 4096, G = 512: the largest tables
])
def test_edge_shapes(N, g, E, S, K, T, d):
    w, topk, gates, table, owner = _custom(N, g, E, S, K, T, d, seed=N * 100 + K)
    check_against_oracle(w, 9, topk, gates, table, owner, step=1)
    check_against_oracle(w, 9, topk, gates, table, owner, step=1, mode=1)


def test_empty_inputs_are_no_ops():
    w = W.WORKLOADS["tiny"]
    table, owner = W.layout(w, 0)
    L = B.cobalt_layout_create(w.N, w.g, w.E, w.S, table, owner)
    e0 = torch.zeros(0, w.K, dtype=torch.int32, device="cuda")
    coact = torch.zeros(w.E, w.E, dtype=torch.int32, device="cuda")
    B.cobalt_coact_stats(e0, w.E, coact, None, B.stats_workspace_for(0, w.K, w.E))
    B.cobalt_assign(L, e0, None, 0, 0, 0, e0.clone())
    counts = torch.full((w.G, w.G), 5, dtype=torch.int32, device="cuda")
    offsets = torch.full((w.G * w.G + 1,), 5, dtype=torch.int64, device="cuda")
    x0 = torch.zeros(0, 64, dtype=torch.bfloat16, device="cuda")
    p0 = torch.zeros(0, 64, dtype=torch.bfloat16, device="cuda")
    B.cobalt_dispatch_pack(e0, None, w.G, x0, counts, offsets, e0.clone(), p0,
                           B.workspace_for(0, w.K, w.G))
    B.cobalt_combine(p0, e0, torch.zeros(0, w.K, device="cuda"), x0.clone())
    torch.cuda.synchronize()
    assert int(coact.abs().sum()) == 0
    assert int(counts.abs().sum()) == 0 and int(offsets.abs().sum()) == 0
    B.cobalt_layout_destroy(L)


def test_index_only_dispatch_matches():
    w = W.with_sizes(W.WORKLOADS["clusters-e64"], T=32 * 77)
    topk, _ = W.routing(w, 1)
    table, owner = W.layout(w, 1)
    L = B.cobalt_layout_create(w.N, w.g, w.E, w.S, table, owner)
    a = torch.empty(w.T, w.K, dtype=torch.int32, device="cuda")
    B.cobalt_assign(L, topk.cuda(), None, 1, 0, 0, a)
    counts = torch.empty(w.G, w.G, dtype=torch.int32, device="cuda")
    offsets = torch.empty(w.G * w.G + 1, dtype=torch.int64, device="cuda")
    pos = torch.empty(w.T, w.K, dtype=torch.int32, device="cuda")
    B.cobalt_dispatch_pack(a, None, w.G, None, counts, offsets, pos, None,
                           B.workspace_for(w.T, w.K, w.G))
    c, o, p, _ = oracle.dispatch(a.cpu().numpy(), w.G)
    assert np.array_equal(pos.cpu().numpy(), p) and np.array_equal(offsets.cpu().numpy(), o)
    B.cobalt_layout_destroy(L)


def test_validate_routing_flags():
    topk = dev_i32([[0, 1], [2, 2], [3, 9]])
    assert B.cobalt_validate_routing(topk, None, 4, 4) == 1 | 2
    src = dev_i32([0, 2, 1])
    assert B.cobalt_validate_routing(topk, src, 16, 4) & 8
    assert B.cobalt_validate_routing(dev_i32([[0, 1], [2, 3]]), dev_i32([0, 3]), 4, 4) == 0
    assert B.cobalt_validate_routing(dev_i32([[0, 1]]), dev_i32([4]), 4, 4) == 4


def test_round_trip_returns_x():
    """expert_out = packed, gates summing to one: y equals x by value."""
    w = W.with_sizes(W.WORKLOADS["colocate-e128"], T=32 * 64, d=1024)
    st = PL.RoutingStep(w, seed=2, device="cuda", expert_out="roundtrip", route_device="cpu")
    st.run()
    torch.cuda.synchronize()
    assert torch.equal(st.y.float(), st.x.float())
    st.close()


@pytest.mark.parametrize("name,T", [("tiny", 4096), ("clusters-e64", 5003), ("drift-e384", 64 * 50),
                                    ("colocate-e256", 64 * 300 + 7)])
def test_replica_load_matches_oracle(name, T):
    """Per-replica task counts w_er (Section 3.1) from the assignment."""
    w = W.with_sizes(W.WORKLOADS[name], T=T)
    topk, _ = W.routing(w, w.seed)
    table, owner = W.layout(w, w.seed)
    src = W.ragged_src(T, w.G, seed=1)
    tabs = oracle.layout_tables(w.N, w.g, w.E, table, owner)
    a, _ = oracle.assign(w.N, w.g, w.E, tabs, topk.numpy(), src, seed=2)
    a[0, 0] = -1  # out-of-range ranks are skipped
    load = torch.zeros(w.E, w.G, dtype=torch.int32, device="cuda")
    ws = B.replica_load_workspace_for(T, w.K, w.E, w.G)
    ws.fill_(0x5A)
    B.cobalt_replica_load(dev_i32(topk.numpy()), dev_i32(a), w.E, w.G, load, ws)
    B.cobalt_replica_load(dev_i32(topk.numpy()), dev_i32(a), w.E, w.G, load, ws)
    ref = oracle.replica_load(topk.numpy(), a, w.E, w.G)
    ref = oracle.replica_load(topk.numpy(), a, w.E, w.G, ref)
    assert np.array_equal(u32(load), ref)


def test_replica_load_uint32_partials():
    """Just over 64 chunks of 65535 pairs: the chunks' counts may pass
    65535, so the partials are uint32 (T * K = 4 194 320, K = 8, E = 256,
    G = 64), with a few pairs out of range."""
    rng = np.random.default_rng(6)
    T, K, E, G = 524290, 8, 256, 64
    topk = rng.integers(0, E, size=(T, K)).astype(np.int32)
    a = rng.integers(0, G, size=(T, K)).astype(np.int32)
    a[rng.random((T, K)) < 1e-4] = G
    load = torch.zeros(E, G, dtype=torch.int32, device="cuda")
    B.cobalt_replica_load(dev_i32(topk), dev_i32(a), E, G, load,
                          B.replica_load_workspace_for(T, K, E, G))
    assert np.array_equal(u32(load), oracle.replica_load(topk, a, E, G))


def test_replica_load_many_bands():
    """E * G beyond one LDS band (E = 4096, G = 32)."""
    rng = np.random.default_rng(4)
    T, K, E, G = 3000, 8, 4096, 32
    topk = rng.integers(0, E, size=(T, K)).astype(np.int32)
    a = rng.integers(0, G, size=(T, K)).astype(np.int32)
    load = torch.zeros(E, G, dtype=torch.int32, device="cuda")
    B.cobalt_replica_load(dev_i32(topk), dev_i32(a), E, G, load,
                          B.replica_load_workspace_for(T, K, E, G))
    assert np.array_equal(u32(load), oracle.replica_load(topk, a, E, G))


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("name,T,d", [("tiny", 4096, 512), ("clusters-e64", 32 * 97, 256),
                                      ("colocate-e256", 64 * 30, 512), ("drift-e384", 64 * 21, 256)])
def test_path_matches_oracle_over_seeds(seed, name, T, d):
    """Every step at seeds 0, 1 and 2 (routing, layout and draws all change
    with the seed), in both assignment modes."""
    w = W.with_sizes(W.WORKLOADS[name], T=T, d=d)
    print(f"seed case {name} seed={seed}", flush=True)
    topk, gates = W.routing(w, seed)
    table, owner = W.layout(w, seed)
    for mode in (0, 1):
        check_against_oracle(w, seed, topk.numpy(), gates.numpy(), table, owner, step=seed,
                             mode=mode)


def test_every_call_is_deterministic_over_ten_repeats():
    """Ten repeats of the four calls (fresh statistics each time) give the
    same bits: a race in the look-back scan, the statistics or the scatter
    would show up as a difference."""
    w = W.with_sizes(W.WORKLOADS["colocate-e256"], T=64 * 300 + 17, d=1024)
    print("determinism case colocate-e256 T=19217 d=1024", flush=True)
    st = PL.RoutingStep(w, seed=7, device="cuda", route_device="cpu",
                        src=W.ragged_src(w.T, w.G, seed=7))
    ref = None
    for rep in range(10):
        st.coact.zero_()
        st.count.zero_()
        st.run()
        torch.cuda.synchronize()
        got = [u32(st.coact), u32(st.count), st.assigned.cpu().numpy(), st.remote.cpu().numpy(),
               st.counts.cpu().numpy(), st.offsets.cpu().numpy(), st.pos.cpu().numpy(),
               PL.bf16_bits(st.packed), PL.bf16_bits(st.y)]
        if ref is None:
            ref = got
        else:
            for a, b in zip(ref, got):
                assert np.array_equal(a, b), f"repeat {rep} differs"
    st.close()


def _random_topk(rng, T, E, K):
    """T tokens of K distinct ids in [0, E), drawn without a T x E matrix."""
    out = np.empty((T, K), np.int32)
    need = np.arange(T)
    draws = rng.integers(0, E, size=(T, K))
    out[:] = draws
    while True:
        s = np.sort(out[need], axis=1)
        dup = (s[:, 1:] == s[:, :-1]).any(1) if K > 1 else np.zeros(len(need), bool)
        need = need[dup]
        if not len(need):
            return out
        out[need] = rng.integers(0, E, size=(len(need), K))


@pytest.mark.parametrize("seed", range(6))
def test_statistics_random_calls(seed):
    """Random (T, E, K) up to T = 400 000 and E = 4096, with a few tokens
    that repeat an id or hold an out-of-range one: the library against the
    oracle on the tokens with ids in range plus the valid-slot brute force
    on the others (the counts add over tokens)."""
    rng = np.random.default_rng(1000 + seed)
    for _ in range(4):
        E = int(rng.choice([3, 16, 64, 255, 256, 384, 1000, 4096]))
        K = int(rng.integers(1, min(16, E) + 1))
        T = int(rng.choice([1, 1023, 4096, 65536, 131077, 262144, 400000]))
        topk = _random_topk(rng, T, E, K)
        bad = np.nonzero(rng.random(T) < 0.002)[0]
        for r in bad:
            if K > 1 and rng.random() < 0.5:
                topk[r, int(rng.integers(1, K))] = topk[r, 0]
            else:
                topk[r, int(rng.integers(0, K))] = int(rng.choice([-1, E, E + 7]))
        good = ((topk >= 0) & (topk < E)).all(1)
        C, cnt = oracle.coact_stats(topk[good], E)
        if (~good).any():
            Cb, cb = _stats_valid_slots(topk[~good], E)
            C = C + Cb
            cnt = cnt + cb
        print(f"statistics seed={seed} T={T} E={E} K={K} odd tokens={len(bad)}", flush=True)
        coact = torch.zeros(E, E, dtype=torch.int32, device="cuda")
        count = torch.zeros(E, dtype=torch.int32, device="cuda")
        B.cobalt_coact_stats(dev_i32(topk), E, coact, count, B.stats_workspace_for(T, K, E))
        assert np.array_equal(u32(coact), C)
        assert np.array_equal(u32(count), cnt)
