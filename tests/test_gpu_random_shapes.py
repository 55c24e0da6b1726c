"""GPU parity on seeded random shapes: every call of the path, and the
node-deduplicated dispatch and node-level combine, on configurations drawn
across the ABI's ranges (1-16 nodes, 1-32 GPUs per node up to 512 ranks,
E up to 4096, K 1-16, 8-4096-element rows, null, contiguous-length and
ragged sources), each checked bit for bit against the oracle."""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import pipeline as PL
from test_gpu_parity import _custom, check_against_oracle

pytestmark = pytest.mark.gpu


def _configs(n, seed=2024):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        N = int(rng.choice([1, 2, 3, 4, 5, 8, 16]))
        g = int(rng.choice([1, 2, 3, 4, 8, 16, 32]))
        G = N * g
        if G > 512:
            continue
        per = int(rng.integers(1, 9))
        E = G * per
        if E > 4096:
            continue
        S = per + int(rng.integers(0, 4))
        K = int(rng.integers(1, min(16, E) + 1))
        srckind = str(rng.choice(["null", "ragged"]))
        m = int(rng.integers(1, 40))
        T = G * m if srckind == "null" else G * m + int(rng.integers(1, G + 1))
        d = 8 * int(rng.choice([1, 2, 3, 5, 16, 64, 129, 256, 512]))
        out.append((N, g, E, S, K, T, d, srckind, int(rng.integers(1 << 30))))
    return out


# COBALT_RANDOM_SHAPES=n,seed draws another set (default: 48 shapes, seed 2024)
_n, _seed = (int(v) for v in os.environ.get("COBALT_RANDOM_SHAPES", "48,2024").split(","))
CONFIGS = _configs(_n, _seed)


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


@pytest.mark.parametrize("N,g,E,S,K,T,d,srckind,seed", CONFIGS,
                         ids=[f"N{c[0]}g{c[1]}E{c[2]}S{c[3]}K{c[4]}T{c[5]}d{c[6]}{c[7]}"
                              for c in CONFIGS])
def test_random_shape(N, g, E, S, K, T, d, srckind, seed):
    print(f"random shape N={N} g={g} E={E} S={S} K={K} T={T} d={d} src={srckind}", flush=True)
    w, topk, gates, table, owner = _custom(N, g, E, S, K, T, d, seed)
    G = N * g
    src = None
    if srckind == "ragged":
        rng = np.random.default_rng(seed + 1)
        src = np.sort(rng.integers(0, G, size=T)).astype(np.int32)
    mode = seed % 2
    check_against_oracle(w, seed, topk, gates, table, owner, src=src, step=seed % 5, mode=mode)

    # the node-deduplicated dispatch and node-level combine of the oracle's assignment
    tabs = oracle.layout_tables(N, g, E, table, owner)
    a, _ = oracle.assign(N, g, E, tabs, topk, src, seed=seed, step=seed % 5, mode=mode)
    _, _, pos, _ = oracle.dispatch(a, G, src)
    gen = torch.Generator().manual_seed(seed + 3)
    x_bits = PL.bf16_bits(torch.randn(T, d, generator=gen).to(torch.bfloat16))
    eo_bits = PL.bf16_bits(torch.randn(T * K, d, generator=gen).to(torch.bfloat16))
    counts, offsets, node_pos, fwd, row_token, packed = oracle.node_dispatch(a, N, g, src, x_bits)
    cap = T * min(K, N)
    rows = int(offsets[-1])
    t_a = dev(a, np.int32)
    t_src = None if src is None else dev(src, np.int32)
    n_counts = torch.empty(G, N, dtype=torch.int32, device="cuda")
    n_offsets = torch.empty(G * N + 1, dtype=torch.int64, device="cuda")
    n_pos = torch.empty(T, N, dtype=torch.int32, device="cuda")
    n_fwd = torch.empty(cap, dtype=torch.int32, device="cuda")
    n_tok = torch.empty(cap, dtype=torch.int32, device="cuda")
    n_packed = torch.empty(cap, d, dtype=torch.bfloat16, device="cuda")
    x = torch.from_numpy(x_bits.view(np.int16)).view(torch.bfloat16).cuda()
    B.cobalt_node_dispatch_pack(t_a, t_src, N, g, x, n_counts, n_offsets, n_pos, n_fwd, n_tok,
                                n_packed, B.node_workspace_for(T, N, g))
    partial = torch.empty(cap, d, dtype=torch.bfloat16, device="cuda")
    y = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
    eo = torch.from_numpy(eo_bits.view(np.int16)).view(torch.bfloat16).cuda()
    B.cobalt_node_combine(eo, dev(pos, np.int32), t_a, dev(gates, np.float32), n_pos, N, g,
                          partial, y)
    torch.cuda.synchronize()
    assert np.array_equal(n_counts.cpu().numpy(), counts)
    assert np.array_equal(n_offsets.cpu().numpy(), offsets)
    assert np.array_equal(n_pos.cpu().numpy(), node_pos)
    assert np.array_equal(n_fwd.cpu().numpy().view(np.uint32)[:rows], fwd)
    assert np.array_equal(n_tok.cpu().numpy()[:rows], row_token)
    assert np.array_equal(PL.bf16_bits(n_packed)[:rows], packed)
    ref_part, ref_y = oracle.node_combine(eo_bits, pos, a, gates, node_pos, g, node_rows=cap)
    assert np.array_equal(PL.bf16_bits(partial)[:rows], ref_part[:rows])
    assert np.array_equal(PL.bf16_bits(y), ref_y)
