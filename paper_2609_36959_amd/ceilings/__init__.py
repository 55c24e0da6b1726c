"""Reference kernels for the benchmark's HBM ceilings (libceilings.so, built
from ceilings.hip): a one-pass streaming read, fill and copy, the pack's
store pattern without its loads, and the combine's row loads without their
fold. Measurement instruments only; the routing library never uses them.
Every function takes torch tensors on the current device and enqueues on
the current stream (or `stream`)."""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libceilings.so")
SRC_PATH = os.path.join(HERE, "ceilings.hip")

_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_36959_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        for name, args in (("ceil_read", [P, i64, P, P]), ("ceil_fill", [P, i64, P]),
                           ("ceil_copy", [P, P, i64, P]),
                           ("ceil_pack_store", [P, i64, i32, i64, P, P]),
                           ("ceil_gather_read", [P, P, i64, i32, i64, P, P]),
                           ("ceil_stream_blocks", [i64])):
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = i64 if name == "ceil_stream_blocks" else ctypes.c_int
        _lib = L
    return _lib


def _s(stream):
    return (torch.cuda.current_stream() if stream is None else stream).cuda_stream


def _ok(name, rc):
    if rc != 0:
        raise RuntimeError(f"{name} failed with status {rc}")


def stream_blocks(nbytes: int) -> int:
    return int(lib().ceil_stream_blocks(nbytes))


def read(buf: torch.Tensor, out: torch.Tensor, stream=None) -> None:
    """XOR of each workgroup's 32-bit words of buf into out
    [stream_blocks(nbytes)]."""
    n = buf.numel() * buf.element_size()
    assert out.dtype in (torch.int32, torch.uint32) and out.numel() >= stream_blocks(n)
    _ok("ceil_read", lib().ceil_read(buf.data_ptr(), n, out.data_ptr(), _s(stream)))


def fill(buf: torch.Tensor, stream=None) -> None:
    _ok("ceil_fill", lib().ceil_fill(buf.data_ptr(), buf.numel() * buf.element_size(), _s(stream)))


def copy(src: torch.Tensor, dst: torch.Tensor, stream=None) -> None:
    n = src.numel() * src.element_size()
    assert dst.numel() * dst.element_size() >= n
    _ok("ceil_copy", lib().ceil_copy(src.data_ptr(), dst.data_ptr(), n, _s(stream)))


def pack_store(pos: torch.Tensor, packed: torch.Tensor, stream=None) -> None:
    T, K = pos.shape
    assert packed.shape[0] == T * K and pos.dtype == torch.int32
    _ok("ceil_pack_store", lib().ceil_pack_store(pos.data_ptr(), T, K, packed.shape[1],
                                                 packed.data_ptr(), _s(stream)))


def gather_read(rows: torch.Tensor, pos: torch.Tensor, out: torch.Tensor, stream=None) -> None:
    """out [T * ceil(d / 1024)] receives each workgroup's XOR."""
    T, K = pos.shape
    d = rows.shape[1]
    assert rows.shape[0] == T * K and out.numel() >= T * ((d // 8 + 127) // 128)
    _ok("ceil_gather_read", lib().ceil_gather_read(rows.data_ptr(), pos.data_ptr(), T, K, d,
                                                   out.data_ptr(), _s(stream)))
