"""Pins of the oracle's bf16 conversions against torch's CPU bfloat16
conversions (a library routine: bf16 is the top half of an fp32, narrowed
with round-to-nearest-even)."""
import numpy as np
import torch

import oracle


def _torch_widen(bits):
    t = torch.from_numpy(bits.astype(np.uint16).view(np.int16)).view(torch.bfloat16)
    return t.float().numpy().view(np.uint32)


def _torch_narrow(vals):
    return torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def test_widen_all_65536_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    mine = oracle.bf16_to_f32(bits).view(np.uint32)
    ref = _torch_widen(bits)
    # a float returned through ctypes becomes a Python double, which quiets
    # signalling NaNs; NaN patterns are compared as NaN, the rest bit for bit
    nan = ((bits & 0x7F80) == 0x7F80) & ((bits & 0x7F) != 0)
    assert np.array_equal(mine[~nan], ref[~nan])
    assert np.all(np.isnan(mine[nan].view(np.float32)))


def test_narrow_random_and_edge_patterns():
    rng = np.random.default_rng(0)
    raw = rng.integers(0, 2**32, size=60000, dtype=np.uint64).astype(np.uint32)
    edges = []
    for hi in (0x0000, 0x0001, 0x3F80, 0x3F81, 0x7F7F, 0x807F, 0xBF80, 0x7F80, 0xFF80):
        for lo in (0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF):
            edges.append((hi << 16) | lo)
    bits = np.concatenate([raw, np.array(edges, np.uint32)])
    vals = bits.view(np.float32)
    mine = oracle.f32_to_bf16(vals)
    ref = _torch_narrow(vals.copy())
    nan = np.isnan(vals)
    assert np.array_equal(mine[~nan], ref[~nan])
    # NaN stays NaN with its sign
    m = mine[nan]
    assert np.all((m & 0x7F80) == 0x7F80) and np.all((m & 0x7F) != 0)
    assert np.array_equal(m >> 15, (bits[nan] >> 31).astype(np.uint16))


def test_round_half_to_even_cases():
    # 1 + 2^-8 lies halfway between bf16 1.0 and 1.0078125: ties to even (1.0)
    cases = {0x3F808000: 0x3F80, 0x3F818000: 0x3F82, 0x3F808001: 0x3F81,
             0x7F7FFFFF: 0x7F80, 0x00008000: 0x0000, 0x00018000: 0x0002}
    for b, want in cases.items():
        v = np.array([b], np.uint32).view(np.float32)
        assert int(oracle.f32_to_bf16(v)[0]) == want
