"""The benchmark's HBM reference kernels do the traffic they are timed for:
each result is checked against numpy, so a ceiling the benchmark reports
comes from a kernel that really read or wrote every byte it counts."""
import numpy as np
import pytest
import torch

from paper_2609_36959_amd import ceilings as C

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    C.lib()
    yield
    torch.cuda.synchronize()


def words(n16, seed):
    rng = np.random.default_rng(seed)
    return rng.integers(0, 2**32, size=n16 * 4, dtype=np.uint64).astype(np.uint32)


@pytest.mark.parametrize("n16", [1, 255, 256, 257, 70001])
def test_fill_copy_read(n16):
    print(f"ceilings n16={n16}", flush=True)
    buf = torch.zeros(n16 * 4, dtype=torch.int32, device="cuda")
    C.fill(buf)
    k = np.arange(n16, dtype=np.uint32)
    want = np.stack([k, k ^ np.uint32(0x9E3779B9), ~k, k * np.uint32(3)], 1).ravel()
    assert np.array_equal(buf.cpu().numpy().view(np.uint32), want)
    src = torch.from_numpy(words(n16, n16).view(np.int32)).cuda()
    dst = torch.zeros_like(src)
    C.copy(src, dst)
    assert torch.equal(src, dst)
    nb = C.stream_blocks(n16 * 16)
    out = torch.zeros(nb, dtype=torch.int32, device="cuda")
    C.read(src, out)
    w = src.cpu().numpy().view(np.uint32)
    pad = np.zeros(nb * 256 * 4, np.uint32)
    pad[: w.size] = w
    want = np.bitwise_xor.reduce(pad.reshape(nb, -1), axis=1)
    assert np.array_equal(out.cpu().numpy().view(np.uint32), want)


@pytest.mark.parametrize("T,K,d", [(300, 8, 1024), (77, 3, 2056), (64, 16, 64), (5, 1, 8)])
def test_pack_store_and_gather_read(T, K, d):
    print(f"ceilings T={T} K={K} d={d}", flush=True)
    rng = np.random.default_rng(T + K + d)
    pos = rng.permutation(T * K).astype(np.int32).reshape(T, K)
    pos_t = torch.from_numpy(pos).cuda()
    packed = torch.zeros(T * K, d, dtype=torch.bfloat16, device="cuda")
    C.pack_store(pos_t, packed)
    got = packed.view(torch.int32).cpu().numpy().view(np.uint32).reshape(T * K, d // 8, 4)
    c = np.arange(d // 8, dtype=np.uint32)
    for t in range(T):
        for j in range(K):
            row = got[pos[t, j]]
            assert np.all(row[:, 0] == t) and np.all(row[:, 1] == j)
            assert np.array_equal(row[:, 2], c) and np.all(row[:, 3] == 0x5A5A5A5A)
    rows_np = words(T * K * d // 8, 7)
    rows = torch.from_numpy(rows_np.view(np.int32)).cuda().view(torch.bfloat16).view(T * K, d)
    groups = (d // 8 + 127) // 128
    out = torch.zeros(T * groups, dtype=torch.int32, device="cuda")
    C.gather_read(rows, pos_t, out)
    r = rows_np.reshape(T * K, d // 8, 4)
    want = np.zeros(T * groups, np.uint32)
    for t in range(T):
        for g in range(groups):
            sl = r[pos[t], g * 128:(g + 1) * 128]
            want[t * groups + g] = np.bitwise_xor.reduce(sl.ravel())
    assert np.array_equal(out.cpu().numpy().view(np.uint32), want)
