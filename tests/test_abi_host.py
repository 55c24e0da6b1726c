"""The C-ABI library on the host (no GPU): it loads, exports every function
include/cobalt.h declares, and rejects bad arguments before touching the
device."""
import ctypes
import re
import subprocess

import numpy as np
import pytest

from paper_2609_36959_amd import binding as B

EINVAL, EUNSUPPORTED, EDATA = 1, 2, 5


def declared_functions():
    src = open(B.HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(cobalt_[a-z_]+)\s*\(", src)))


def test_header_declares_the_path():
    names = declared_functions()
    for required in ("cobalt_coact_stats", "cobalt_assign", "cobalt_dispatch_pack",
                     "cobalt_combine", "cobalt_layout_create", "cobalt_layout_destroy"):
        assert required in names


def test_library_exports_every_declared_function():
    L = B.lib()
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    for name in declared_functions():
        assert name in exported, name
        assert getattr(L, name) is not None
    # and exports nothing else under the cobalt_ prefix
    assert {n for n in exported if n.startswith("cobalt_")} == set(declared_functions())


def test_status_strings():
    L = B.lib()
    for s in range(6):
        assert L.cobalt_status_string(s)
    assert L.cobalt_status_string(0) == b"ok"


def test_workspace_size_query():
    L = B.lib()
    s3 = L.cobalt_coact_stats_workspace_bytes(131072, 8, 256)
    # one 32-bit partial histogram of the pair triangle per 2048-token chunk
    assert s3 >= 64 * 256 * 255 // 2 * 4 and s3 % 256 == 0
    assert L.cobalt_coact_stats_workspace_bytes(100, 2, 4096) > 0
    assert L.cobalt_coact_stats_workspace_bytes(100, 2, 4097) == 0
    a = L.cobalt_dispatch_workspace_bytes(131072, 8, 64)
    b = L.cobalt_dispatch_workspace_bytes(4096, 2, 8)
    assert a > b > 0 and a % 256 == 0
    assert L.cobalt_dispatch_workspace_bytes(-1, 8, 64) == 0
    assert L.cobalt_dispatch_workspace_bytes(10, 17, 64) == 0
    assert L.cobalt_dispatch_workspace_bytes(10, 8, 513) == 0
    n1 = L.cobalt_node_dispatch_workspace_bytes(131072, 8, 8)
    n2 = L.cobalt_node_dispatch_workspace_bytes(4096, 2, 4)
    assert n1 > n2 > 0 and n1 % 256 == 0
    assert L.cobalt_node_dispatch_workspace_bytes(10, 17, 1) == 0
    assert L.cobalt_node_dispatch_workspace_bytes(10, 2, 33) == 0
    assert L.cobalt_node_dispatch_workspace_bytes(-1, 2, 4) == 0


def _p(v):
    return ctypes.c_void_p(v)


def test_argument_checks_reject_before_device_work():
    L = B.lib()
    fake = _p(4096)  # never dereferenced: every call below fails its host checks
    # coact_stats: null output, K out of range, E out of range
    big = 1 << 40
    assert L.cobalt_coact_stats(fake, 10, 2, 16, None, None, fake, big, None) == EINVAL
    assert L.cobalt_coact_stats(fake, 10, 17, 16, fake, None, fake, big, None) == EINVAL
    assert L.cobalt_coact_stats(fake, 10, 2, 0, fake, None, fake, big, None) == EINVAL
    assert L.cobalt_coact_stats(fake, 10, 2, 16, fake, None, None, big, None) == EINVAL
    assert L.cobalt_coact_stats(fake, 10, 2, 16, fake, None, _p(4100), big, None) == EINVAL
    assert L.cobalt_coact_stats(fake, 10, 2, 16, fake, None, fake, 16, None) == EINVAL
    assert L.cobalt_coact_stats(fake, 1 << 28, 8, 16, fake, None, fake, big,
                                None) == EUNSUPPORTED
    # K > E: a token cannot select K distinct experts
    assert L.cobalt_coact_stats(fake, 10, 5, 4, fake, None, fake, big, None) == EINVAL
    # assign: null layout, bad mode
    assert L.cobalt_assign(None, fake, None, 8, 2, 0, 0, 0, fake, None, None) == EINVAL
    assert L.cobalt_assign(fake, fake, None, 8, 2, 0, 0, 7, fake, None, None) == EINVAL
    # dispatch: x without packed, d not a multiple of 8, misaligned workspace
    args = [fake, None, 8, 2, 4]
    assert L.cobalt_dispatch_pack(*args, fake, 8, fake, fake, fake, None, fake, 1 << 20,
                                  None) == EINVAL
    assert L.cobalt_dispatch_pack(*args, fake, 12, fake, fake, fake, fake, fake, 1 << 20,
                                  None) == EINVAL
    assert L.cobalt_dispatch_pack(*args, None, 0, fake, fake, fake, None, _p(4100), 1 << 20,
                                  None) == EINVAL
    assert L.cobalt_dispatch_pack(*args, None, 0, fake, fake, fake, None, fake, 16,
                                  None) == EINVAL  # workspace too small
    assert L.cobalt_dispatch_pack(fake, None, 9, 2, 4, None, 0, fake, fake, fake, None, fake,
                                  1 << 20, None) == EINVAL  # T % G != 0 without src_rank
    # workspace-free dispatch: the same checks, and sizes whose workspace
    # exceeds the fixed scratch are refused before any device work
    assert L.cobalt_dispatch_pack_noalloc(*args, fake, 8, fake, fake, fake, None,
                                          None) == EINVAL
    assert L.cobalt_dispatch_pack_noalloc(*args, fake, 12, fake, fake, fake, fake,
                                          None) == EINVAL
    assert L.cobalt_dispatch_pack_noalloc(fake, None, 9, 2, 4, None, 0, fake, fake, fake, None,
                                          None) == EINVAL
    cap = B.DISPATCH_NOALLOC_SCRATCH_BYTES
    assert L.cobalt_dispatch_workspace_bytes(66973696, 1, 64) <= cap
    assert L.cobalt_dispatch_workspace_bytes(66973696 + 4096, 1, 64) > cap
    assert L.cobalt_dispatch_pack_noalloc(fake, None, 66973696 // 8 + 256, 8, 64, None, 0, fake,
                                          fake, fake, None, None) == EUNSUPPORTED
    assert L.cobalt_dispatch_pack_noalloc(fake, None, 1800 * 512, 8, 512, None, 0, fake,
                                          fake, fake, None, None) == EUNSUPPORTED
    # node dispatch: x without packed, null forwarding index, N or g out of
    # range, misaligned or short workspace, T % G != 0 without src_rank
    nargs = [fake, None, 8, 2, 2, 2]
    assert L.cobalt_node_dispatch_pack(*nargs, fake, 8, fake, fake, fake, fake, None, None, fake,
                                       1 << 20, None) == EINVAL
    assert L.cobalt_node_dispatch_pack(*nargs, None, 0, fake, fake, fake, None, None, None, fake,
                                       1 << 20, None) == EINVAL
    assert L.cobalt_node_dispatch_pack(fake, None, 8, 2, 17, 1, None, 0, fake, fake, fake, fake,
                                       None, None, fake, 1 << 20, None) == EINVAL
    assert L.cobalt_node_dispatch_pack(fake, None, 8, 2, 2, 33, None, 0, fake, fake, fake, fake,
                                       None, None, fake, 1 << 20, None) == EINVAL
    assert L.cobalt_node_dispatch_pack(*nargs, None, 0, fake, fake, fake, fake, None, None,
                                       _p(4100), 1 << 20, None) == EINVAL
    assert L.cobalt_node_dispatch_pack(*nargs, None, 0, fake, fake, fake, fake, None, None, fake,
                                       16, None) == EINVAL
    assert L.cobalt_node_dispatch_pack(fake, None, 9, 2, 2, 2, None, 0, fake, fake, fake, fake,
                                       None, None, fake, 1 << 20, None) == EINVAL
    # EMA: decay outside [0, 1] or NaN, unknown flags, null counts, E out of range
    f = ctypes.c_float
    assert L.cobalt_coact_ema(fake, fake, 8, f(1.5), 0, fake, None, None, None) == EINVAL
    assert L.cobalt_coact_ema(fake, fake, 8, f(float("nan")), 0, fake, None, None,
                              None) == EINVAL
    assert L.cobalt_coact_ema(fake, fake, 8, f(0.5), 4, fake, None, None, None) == EINVAL
    assert L.cobalt_coact_ema(None, fake, 8, f(0.5), 0, fake, None, None, None) == EINVAL
    assert L.cobalt_coact_ema(fake, fake, 4097, f(0.5), 0, fake, None, None, None) == EINVAL
    assert L.cobalt_count_ema(fake, 10, f(-0.5), 0, fake, None) == EINVAL
    assert L.cobalt_count_ema(None, 10, f(0.5), 0, fake, None) == EINVAL
    assert L.cobalt_count_ema(fake, -1, f(0.5), 0, fake, None) == EINVAL
    assert L.cobalt_count_ema(None, 0, f(0.5), 2, None, None) == 0  # nothing to do
    # combine: d not a multiple of 8, misaligned rows
    assert L.cobalt_combine(fake, fake, fake, 8, 2, 12, fake, None, None) == EINVAL
    assert L.cobalt_combine(_p(4098), fake, fake, 8, 2, 16, fake, None, None) == EINVAL
    # node combine: null node_pos, d not a multiple of 8, N or g out of range,
    # misaligned partial rows, T = 0 does nothing
    cargs = [fake, fake, fake, fake]
    assert L.cobalt_node_combine(*cargs, None, 8, 2, 2, 2, 16, fake, fake, None) == EINVAL
    assert L.cobalt_node_combine(*cargs, fake, 8, 2, 2, 2, 12, fake, fake, None) == EINVAL
    assert L.cobalt_node_combine(*cargs, fake, 8, 2, 17, 2, 16, fake, fake, None) == EINVAL
    assert L.cobalt_node_combine(*cargs, fake, 8, 2, 2, 33, 16, fake, fake, None) == EINVAL
    assert L.cobalt_node_combine(*cargs, fake, 8, 2, 2, 2, 16, _p(4104), fake, None) == EINVAL
    assert L.cobalt_node_combine(None, None, None, None, None, 0, 2, 2, 2, 16, None, None,
                                 None) == 0


def test_layout_create_rejects_invalid_layouts_on_the_host(fig1):
    L = B.lib()
    N, g, E, S = fig1["N"], fig1["g"], fig1["E"], fig1["S"]

    def create(table, owner=None):
        t = np.ascontiguousarray(table, np.int32)
        o = None if owner is None else np.ascontiguousarray(owner, np.int32)
        h = ctypes.c_void_p()
        return L.cobalt_layout_create(N, g, E, S, t.ctypes.data_as(ctypes.c_void_p),
                                      None if o is None else o.ctypes.data_as(ctypes.c_void_p),
                                      ctypes.byref(h))

    t = fig1["table"].copy()
    t[3, 0] = -1
    assert create(t) == EDATA            # d uncovered (Eq. 2 coverage)
    t = fig1["table"].copy()
    t[0, 1] = 0
    assert create(t) == EDATA            # a twice on one rank
    t = fig1["table"].copy()
    t[1, 1] = 9
    assert create(t) == EDATA            # id out of range
    assert create(fig1["table"], [0, 1, 1, 3]) == EDATA  # owner does not hold b
    h = ctypes.c_void_p()
    tt = fig1["table"]
    assert L.cobalt_layout_create(17, 1, E, S, tt.ctypes.data_as(ctypes.c_void_p), None,
                                  ctypes.byref(h)) == EINVAL
    assert L.cobalt_layout_create(N, 33, E, S, tt.ctypes.data_as(ctypes.c_void_p), None,
                                  ctypes.byref(h)) == EINVAL


def test_binding_has_the_c_names():
    for name in declared_functions():
        if name == "cobalt_status_string":
            continue
        assert hasattr(B, name), name


def test_python_layer_calls_no_oracle():
    """The product package never imports the oracle."""
    import glob
    import os
    pat = re.compile(r"^\s*(import\s+oracle|from\s+oracle\b|.*liboracle)", re.M)
    for f in glob.glob(os.path.join(os.path.dirname(B.__file__), "*.py")):
        assert not pat.search(open(f).read()), f
