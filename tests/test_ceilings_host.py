"""The benchmark's reference-kernel library builds for gfx950, exports its
entry points and refuses bad sizes on the host (no GPU needed)."""
import ctypes

from paper_2609_36959_amd import ceilings as C


def test_exports_and_host_checks():
    L = C.lib()
    for name in ("ceil_read", "ceil_fill", "ceil_copy", "ceil_pack_store", "ceil_gather_read"):
        assert getattr(L, name) is not None
    fake = ctypes.c_void_p(4096)
    assert L.ceil_fill(fake, 24, None) == 1          # not a multiple of 16 bytes
    assert L.ceil_read(None, 1024, fake, None) == 1
    assert L.ceil_copy(fake, fake, 0, None) == 1
    assert L.ceil_pack_store(fake, 10, 17, 64, fake, None) == 1   # K > 16
    assert L.ceil_pack_store(fake, 10, 8, 12, fake, None) == 1    # d % 8
    assert L.ceil_gather_read(fake, fake, 10, 8, 16392, fake, None) == 1  # d > 16384
    assert C.stream_blocks(4096 * 16) == 16
