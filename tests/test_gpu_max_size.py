"""The dispatch and combine at the ABI's largest pair count: T*K = 2 147 483 136
pairs (just under 2^31) over 64 ranks, 16-byte rows. Every pos is compared
with the oracle's; packed rows and combined tokens on seeded samples.

It needs about 100 GB of device memory and 30 GB of host memory, and takes
about 15 s on an MI355X. COBALT_SKIP_MAX_SIZE=1 skips it on machines with
less memory."""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import pipeline as PL

def normal_bf16(rows, d, gen, chunk=1 << 26):
    """N(0,1) rows rounded to bf16, drawn in chunks to bound the fp32 staging."""
    out = torch.empty(rows, d, dtype=torch.bfloat16, device="cuda")
    for r0 in range(0, rows, chunk):
        r1 = min(rows, r0 + chunk)
        out[r0:r1] = torch.randn(r1 - r0, d, device="cuda", generator=gen).to(torch.bfloat16)
    return out


pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(os.environ.get("COBALT_SKIP_MAX_SIZE") == "1",
                                 reason="COBALT_SKIP_MAX_SIZE=1 (it needs about 100 GB of HBM)")]


def test_dispatch_and_combine_at_the_largest_pair_count():
    torch.cuda.set_device(0)
    B.lib()
    G, K, d = 64, 8, 8
    T = ((2**31 - 1) // K) // G * G          # null src_rank needs T % G == 0
    TK = T * K
    assert TK < 2**31 and TK > 2**31 - 1024
    print(f"max size: T={T} K={K} pairs={TK}", flush=True)
    gen = torch.Generator(device="cuda").manual_seed(5)
    assigned = torch.randint(0, G, (T, K), dtype=torch.int32, device="cuda", generator=gen)
    x = normal_bf16(T, d, gen)
    counts = torch.empty(G, G, dtype=torch.int32, device="cuda")
    offsets = torch.empty(G * G + 1, dtype=torch.int64, device="cuda")
    pos = torch.empty(T, K, dtype=torch.int32, device="cuda")
    packed = torch.empty(TK, d, dtype=torch.bfloat16, device="cuda")
    B.cobalt_dispatch_pack(assigned, None, G, x, counts, offsets, pos, packed,
                           B.workspace_for(T, K, G))
    torch.cuda.synchronize()
    print("max size: dispatch done", flush=True)
    assert int(offsets[-1].item()) == TK
    assert int(pos.min().item()) == 0 and int(pos.max().item()) == TK - 1

    a_host = assigned.cpu().numpy()
    ref_counts, ref_offsets, ref_pos, _ = oracle.dispatch(a_host, G)
    print("max size: oracle done", flush=True)
    assert np.array_equal(counts.cpu().numpy(), ref_counts)
    assert np.array_equal(offsets.cpu().numpy(), ref_offsets)
    assert np.array_equal(pos.cpu().numpy(), ref_pos), "pos differs"
    del a_host

    rng = np.random.default_rng(5)
    p = rng.choice(TK, size=1 << 20, replace=False)
    rows = torch.from_numpy(ref_pos.ravel()[p].astype(np.int64)).cuda()
    toks = torch.from_numpy(p // K).cuda()
    assert torch.equal(packed[rows].view(torch.int16), x[toks].view(torch.int16))
    del packed, assigned
    torch.cuda.empty_cache()

    # combine over the same rows, stand-in expert outputs, sampled tokens
    eo = normal_bf16(TK, d, gen)
    gates = torch.rand(T, K, device="cuda", generator=gen)
    y = torch.empty(T, d, dtype=torch.bfloat16, device="cuda")
    B.cobalt_combine(eo, pos, gates, y)
    torch.cuda.synchronize()
    print("max size: combine done", flush=True)
    t = np.sort(rng.choice(T, size=1 << 16, replace=False))
    sel = torch.from_numpy(ref_pos[t].ravel().astype(np.int64)).cuda()
    eo_rows = PL.bf16_bits(eo[sel])
    ident = np.arange(len(t) * K, dtype=np.int32).reshape(len(t), K)
    y_ref, _ = oracle.combine(eo_rows, ident, gates.cpu().numpy()[t])
    assert np.array_equal(PL.bf16_bits(y[torch.from_numpy(t).cuda()]), y_ref)
    # hand the memory back before the tests that follow
    del eo, gates, y, pos, x, rows, toks, sel
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
