"""Kernels over tokens are launched over token ranges, since a dispatch
packet holds the grid size in work-items as a 32-bit value. With the limit
lowered through COBALT_MAX_LAUNCH_ITEMS, ordinary sizes run as dozens of
ranges per call, and every output of the per-pair and node-deduplicated
dispatch and combine still equals the oracle's bit for bit (the scatter
and fold, the fan-out copy and combine_kernel for wide rows, and the node
kernels)."""
import contextlib
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import pipeline as PL
from test_gpu_parity import _custom, check_against_oracle

pytestmark = pytest.mark.gpu


@contextlib.contextmanager
def launch_limit(items):
    old = os.environ.get("COBALT_MAX_LAUNCH_ITEMS")
    os.environ["COBALT_MAX_LAUNCH_ITEMS"] = str(items)
    try:
        yield
    finally:
        if old is None:
            del os.environ["COBALT_MAX_LAUNCH_ITEMS"]
        else:
            os.environ["COBALT_MAX_LAUNCH_ITEMS"] = old


def dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a, dtype)).cuda()


def check_node_paths(N, g, K, T, d, a, pos, gates, seed):
    gen = torch.Generator().manual_seed(seed)
    x_bits = PL.bf16_bits(torch.randn(T, d, generator=gen).to(torch.bfloat16))
    eo_bits = PL.bf16_bits(torch.randn(T * K, d, generator=gen).to(torch.bfloat16))
    counts, offsets, node_pos, fwd, row_token, packed = oracle.node_dispatch(a, N, g, None, x_bits)
    G, cap, rows = N * g, T * min(K, N), int(offsets[-1])
    n_counts = torch.empty(G, N, dtype=torch.int32, device="cuda")
    n_offsets = torch.empty(G * N + 1, dtype=torch.int64, device="cuda")
    n_pos = torch.empty(T, N, dtype=torch.int32, device="cuda")
    n_fwd = torch.empty(cap, dtype=torch.int32, device="cuda")
    n_packed = torch.empty(cap, d, dtype=torch.bfloat16, device="cuda")
    x = torch.from_numpy(x_bits.view(np.int16)).view(torch.bfloat16).cuda()
    t_a = dev(a, np.int32)
    B.cobalt_node_dispatch_pack(t_a, None, N, g, x, n_counts, n_offsets, n_pos, n_fwd, None,
                                n_packed, B.node_workspace_for(T, N, g))
    partial = torch.empty(cap, d, dtype=torch.bfloat16, device="cuda")
    y = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
    eo = torch.from_numpy(eo_bits.view(np.int16)).view(torch.bfloat16).cuda()
    B.cobalt_node_combine(eo, dev(pos, np.int32), t_a, dev(gates, np.float32), n_pos, N, g,
                          partial, y)
    torch.cuda.synchronize()
    assert np.array_equal(n_pos.cpu().numpy(), node_pos)
    assert np.array_equal(PL.bf16_bits(n_packed)[:rows], packed)
    ref_part, ref_y = oracle.node_combine(eo_bits, pos, a, gates, node_pos, g, node_rows=cap)
    assert np.array_equal(PL.bf16_bits(partial)[:rows], ref_part[:rows])
    assert np.array_equal(PL.bf16_bits(y), ref_y)


@pytest.mark.parametrize("limit", [1 << 16, 1 << 20])
@pytest.mark.parametrize("N,g,E,S,K,T,d", [
    (8, 8, 256, 5, 8, 64 * 33, 2048),    # scatter and fold, several slices
    (2, 4, 16, 4, 4, 8 * 40, 16392),     # 17 slices: fan-out copy, combine_kernel, node kernels' run-time count
    (4, 8, 64, 3, 1, 32 * 50, 8),        # K = 1, 16-byte rows
])
def test_split_launches_match_the_oracle(limit, N, g, E, S, K, T, d):
    print(f"launch ranges: limit={limit} N={N} g={g} K={K} T={T} d={d}", flush=True)
    w, topk, gates, table, owner = _custom(N, g, E, S, K, T, d, seed=limit % 97 + K)
    with launch_limit(limit):
        check_against_oracle(w, 3, topk, gates, table, owner)
        tabs = oracle.layout_tables(N, g, E, table, owner)
        a, _ = oracle.assign(N, g, E, tabs, topk, None, seed=3)
        _, _, pos, _ = oracle.dispatch(a, N * g)
        check_node_paths(N, g, K, T, d, a, pos, gates, seed=limit % 89)
