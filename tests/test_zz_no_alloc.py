"""The workspace-free dispatch (cobalt_dispatch_pack_noalloc) against the
dispatch with a caller workspace (cobalt_dispatch_pack), through the C ABI:
counts, offsets, pos and packed rows bit for bit, on calls in a row whose
sizes shrink (so a call that read state left by the previous one would
differ), with null and ragged source ranks, a layout-only call near the
scratch limit, and a check against the oracle on the first call."""
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


def _inputs(T, K, G, d, src_kind, seed):
    rng = np.random.default_rng(seed)
    # skewed destinations (density falling with the rank), so buckets differ
    # widely in size
    a = np.minimum((rng.random((T, K), dtype=np.float32) ** 3 * G).astype(np.int32), G - 1)
    src = None if src_kind == "null" else W.ragged_src(T, G, seed)
    x = None
    if d:
        g = torch.Generator().manual_seed(seed)
        x = torch.randn(T, d, generator=g).to(torch.bfloat16).cuda()
    return a, src, x


def _run(entry, a, src, x, G):
    T, K = a.shape
    d = 0 if x is None else x.shape[1]
    t_a = torch.from_numpy(a).cuda()
    t_src = None if src is None else torch.from_numpy(np.ascontiguousarray(src, np.int32)).cuda()
    counts = torch.full((G, G), -1, dtype=torch.int32, device="cuda")
    offsets = torch.full((G * G + 1,), -1, dtype=torch.int64, device="cuda")
    pos = torch.full((T, K), -1, dtype=torch.int32, device="cuda")
    packed = None if x is None else torch.zeros(T * K, d, dtype=torch.bfloat16, device="cuda")
    if entry == "noalloc":
        B.cobalt_dispatch_pack_noalloc(t_a, t_src, G, x, counts, offsets, pos, packed)
    else:
        ws = B.workspace_for(T, K, G)
        ws.fill_(0x5A)
        B.cobalt_dispatch_pack(t_a, t_src, G, x, counts, offsets, pos, packed, ws)
    torch.cuda.synchronize()
    return (counts.cpu().numpy(), offsets.cpu().numpy(), pos.cpu().numpy(),
            None if packed is None else PL.bf16_bits(packed))


def _same(got, ref):
    for g, r in zip(got, ref):
        if r is None:
            assert g is None
        else:
            assert np.array_equal(g, r)


# calls in a row, each smaller than the one before
CALLS = [
    (16384, 6, 32, 2048, "null"),    # 4 x 8 ranks, 24 tiles of look-back state per column
    (3001, 2, 8, 512, "ragged"),     # fewer tiles and columns, ragged tail
    (64, 1, 1, 8, "null"),           # one rank, one tile
]


def test_noalloc_matches_workspace_dispatch_on_shrinking_calls():
    for i, (T, K, G, d, src_kind) in enumerate(CALLS):
        print(f"noalloc call {i}: T={T} K={K} G={G} d={d} src={src_kind}", flush=True)
        a, src, x = _inputs(T, K, G, d, src_kind, seed=100 + i)
        got = _run("noalloc", a, src, x, G)
        ref = _run("workspace", a, src, x, G)
        _same(got, ref)
        if i == 0:
            xb = PL.bf16_bits(x)
            _same(got, oracle.dispatch(a, G, src, xb))
    # and the first call again, after the smaller ones
    T, K, G, d, src_kind = CALLS[0]
    a, src, x = _inputs(T, K, G, d, src_kind, seed=100)
    _same(_run("noalloc", a, src, x, G), _run("workspace", a, src, x, G))


def test_noalloc_layout_only_near_the_scratch_limit():
    # G = 512: the scratch holds the look-back state of up to 7 335 936 pairs
    G, K = 512, 8
    T = 7335936 // K // G * G
    assert B.cobalt_dispatch_workspace_bytes(T, K, G) <= B.DISPATCH_NOALLOC_SCRATCH_BYTES
    print(f"noalloc layout-only call: T={T} K={K} G={G}", flush=True)
    a, src, _ = _inputs(T, K, G, 0, "null", seed=7)
    _same(_run("noalloc", a, src, None, G), _run("workspace", a, src, None, G))
    # then a small call with rows
    a, src, x = _inputs(4096, 2, 8, 512, "null", seed=8)
    _same(_run("noalloc", a, src, x, 8), _run("workspace", a, src, x, 8))


def test_noalloc_rejects_sizes_beyond_the_scratch():
    G, K = 64, 8
    T = (66973696 // K // G + 64) * G
    assert B.cobalt_dispatch_workspace_bytes(T, K, G) > B.DISPATCH_NOALLOC_SCRATCH_BYTES
    a = torch.zeros(T, K, dtype=torch.int32, device="cuda")
    counts = torch.zeros(G, G, dtype=torch.int32, device="cuda")
    offsets = torch.zeros(G * G + 1, dtype=torch.int64, device="cuda")
    pos = torch.zeros(T, K, dtype=torch.int32, device="cuda")
    with pytest.raises(B.CobaltError) as e:
        B.cobalt_dispatch_pack_noalloc(a, None, G, None, counts, offsets, pos, None)
    assert e.value.status == 2  # COBALT_EUNSUPPORTED
    torch.cuda.synchronize()
    assert int(counts.abs().sum()) == 0  # nothing was enqueued
