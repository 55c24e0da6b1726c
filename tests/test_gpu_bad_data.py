"""The hot calls on invalid routing data (ids outside [0, E), ranks outside
[0, G), sources outside [0, G) or out of order). The header leaves their
results unspecified except for what this checks: nothing is written out of
bounds (every output and guard row keeps its sentinel), pairs with an
invalid id or source get rank -1 and pos -1, only valid pairs are placed,
and the rows they get lie inside the placed range. Every index the kernels
take from data is range-checked before use, so these inputs cannot reach
memory outside the buffers."""
import numpy as np
import pytest
import torch

from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import workload as W

pytestmark = pytest.mark.gpu

GUARD = 4096  # elements of sentinel after every output


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    B.lib()
    yield
    torch.cuda.synchronize()


def guarded(shape, dtype, fill):
    """A buffer with GUARD sentinel elements behind it; returns (view, whole)."""
    n = int(np.prod(shape))
    whole = torch.full((n + GUARD,), fill, dtype=dtype, device="cuda")
    return whole[:n].view(*shape), whole


def intact(whole, n, fill):
    tail = whole[n:]
    return bool((tail == fill).all().item()) if tail.dtype != torch.bfloat16 else \
        bool((tail.view(torch.int16) == torch.tensor(fill, dtype=torch.bfloat16).view(torch.int16)).all().item())


@pytest.mark.parametrize("src_kind", ["ragged", "shuffled"])
def test_invalid_ids_ranks_and_sources(src_kind):
    w = W.with_sizes(W.WORKLOADS["clusters-e64"], T=2048 + 29, d=256)
    T, K, E, G, d = w.T, w.K, w.E, w.G, w.d
    rng = np.random.default_rng(3)
    topk = W.routing(w, w.seed)[0].numpy().copy()
    bad_id = rng.random((T, K)) < 0.1
    topk[bad_id] = rng.choice([-7, -1, E, E + 100], size=int(bad_id.sum()))
    src = W.ragged_src(T, G, seed=5)
    if src_kind == "shuffled":
        src = rng.permutation(src)
    bad_src = rng.random(T) < 0.05
    src[bad_src] = rng.choice([-1, G, G + 3], size=int(bad_src.sum()))
    t_topk = torch.from_numpy(topk.astype(np.int32)).cuda()
    t_src = torch.from_numpy(src.astype(np.int32)).cuda()
    flags = B.cobalt_validate_routing(t_topk, t_src, E, G)
    assert flags & 1 and flags & 4 and (src_kind == "ragged" or flags & 8)

    table, owner = W.layout(w, w.seed)
    L = B.cobalt_layout_create(w.N, w.g, E, w.S, table, owner)

    coact, coact_w = guarded((E, E), torch.int32, 0)
    count, count_w = guarded((E,), torch.int32, 0)
    B.cobalt_coact_stats(t_topk, E, coact, count, B.stats_workspace_for(T, K, E))
    assigned, assigned_w = guarded((T, K), torch.int32, -9)
    remote, remote_w = guarded((T,), torch.int16, -9)
    B.cobalt_assign(L, t_topk, t_src, 1, 0, 0, assigned, remote)

    x = torch.randn(T, d, device="cuda").to(torch.bfloat16)
    counts, counts_w = guarded((G, G), torch.int32, -9)
    offsets, offsets_w = guarded((G * G + 1,), torch.int64, -9)
    pos, pos_w = guarded((T, K), torch.int32, -9)
    packed, packed_w = guarded((T * K, d), torch.bfloat16, 0.5)
    B.cobalt_dispatch_pack(assigned, t_src, G, x, counts, offsets, pos, packed,
                           B.workspace_for(T, K, G))
    eo = torch.randn(T * K, d, device="cuda").to(torch.bfloat16)
    gates = torch.rand(T, K, device="cuda")
    y, y_w = guarded((T, d), torch.bfloat16, 0.5)
    B.cobalt_combine(eo, pos, gates, y)
    N, g = w.N, w.g
    cap = T * min(K, N)
    ncounts, ncounts_w = guarded((G, N), torch.int32, -9)
    noffsets, noffsets_w = guarded((G * N + 1,), torch.int64, -9)
    npos, npos_w = guarded((T, N), torch.int32, -9)
    fwd, fwd_w = guarded((cap,), torch.int32, -9)
    rtok, rtok_w = guarded((cap,), torch.int32, -9)
    npacked, npacked_w = guarded((cap, d), torch.bfloat16, 0.5)
    B.cobalt_node_dispatch_pack(assigned, t_src, N, g, x, ncounts, noffsets, npos,
                                fwd, rtok, npacked,
                                B.node_workspace_for(T, N, g))
    load, load_w = guarded((E, G), torch.int32, 0)
    B.cobalt_replica_load(t_topk, assigned, E, G, load,
                          B.replica_load_workspace_for(T, K, E, G))
    torch.cuda.synchronize()

    for v, wbuf, fill in ((coact, coact_w, 0), (count, count_w, 0), (assigned, assigned_w, -9),
                          (remote, remote_w, -9), (counts, counts_w, -9),
                          (offsets, offsets_w, -9), (pos, pos_w, -9), (packed, packed_w, 0.5),
                          (y, y_w, 0.5), (load, load_w, 0), (ncounts, ncounts_w, -9),
                          (noffsets, noffsets_w, -9), (npos, npos_w, -9), (fwd, fwd_w, -9),
                          (rtok, rtok_w, -9), (npacked, npacked_w, 0.5)):
        assert intact(wbuf, v.numel(), fill), "a write past the end of an output"

    a = assigned.cpu().numpy()
    invalid = bad_id | bad_src[:, None]
    assert np.all(a[invalid] == -1)
    assert np.all((a[~invalid] >= 0) & (a[~invalid] < G))
    placed = int(offsets[-1].item())
    assert placed == int((~invalid).sum()) == int(counts.sum().item())
    p = pos.cpu().numpy()
    assert np.all(p[invalid] == -1)
    assert np.all((p[~invalid] >= 0) & (p[~invalid] < placed))
    if src_kind == "ragged":  # in order: the layout is still a permutation
        assert np.array_equal(np.sort(p[~invalid]), np.arange(placed))
    assert torch.isfinite(y.float()).all()
    assert int(count.sum().item()) == int((~bad_id).sum())
    assert int(load.sum().item()) == int((~invalid).sum())

    # node rows: one per (token, node) that a valid pair of the token reaches
    reach = np.zeros((T, N), bool)
    for j in range(K):
        ok = ~invalid[:, j]
        reach[np.nonzero(ok)[0], a[ok, j] // g] = True
    rows = int(noffsets[-1].item())
    assert rows == int(reach.sum()) == int(ncounts.sum().item())
    q = npos.cpu().numpy()
    assert np.all(q[~reach] == -1)
    assert np.all((q[reach] >= 0) & (q[reach] < rows))
    if src_kind == "ragged":
        assert np.array_equal(np.sort(q[reach]), np.arange(rows))
        rt = rtok.cpu().numpy()[:rows]
        assert np.array_equal(rt[q[reach]], np.nonzero(reach)[0])
    B.cobalt_layout_destroy(L)


def test_assign_rejects_k_above_the_layouts_experts():
    """A token selects K distinct experts, so K > E is refused on the host
    and nothing is written."""
    N, g, E, S = 2, 2, 4, 2
    table = np.array([[0, 1], [1, 2], [2, 3], [3, 0]], np.int32)
    L = B.cobalt_layout_create(N, g, E, S, table)
    T, K = 8, 5
    topk = torch.zeros(T, K, dtype=torch.int32, device="cuda")
    out = torch.full((T, K), -3, dtype=torch.int32, device="cuda")
    with pytest.raises(B.CobaltError) as e:
        B.cobalt_assign(L, topk, None, 0, 0, 0, out)
    assert e.value.status == 1  # COBALT_EINVAL
    torch.cuda.synchronize()
    assert bool((out == -3).all().item())
    B.cobalt_layout_destroy(L)
