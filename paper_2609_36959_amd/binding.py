"""Python binding of libcobalt.so (the C ABI in include/cobalt.h).

Argument marshalling only: every function has the name of the C entry point
it calls, takes torch tensors on the current HIP device (memory and streams
come from PyTorch), checks dtypes and shapes, and passes raw pointers. All
work happens in the library's HIP kernels. If the library has not been
built, every call raises; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libcobalt.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "cobalt.h")

STATUS = {0: "COBALT_OK", 1: "COBALT_EINVAL", 2: "COBALT_EUNSUPPORTED", 3: "COBALT_ENOMEM",
          4: "COBALT_EHIP", 5: "COBALT_EDATA"}


class CobaltError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn}: {STATUS.get(status, status)}")


_lib = None


def lib() -> ctypes.CDLL:
    """Load libcobalt.so once, after torch so that both share torch's HIP
    runtime (two runtimes in one process could not share streams)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2609_36959_amd.build` (no fallback exists)")
    L = ctypes.CDLL(LIB_PATH)
    with open("/proc/self/maps") as f:
        runtimes = {ln.split()[-1] for ln in f if "libamdhip64" in ln}
    if len(runtimes) > 1:
        raise RuntimeError(f"more than one HIP runtime mapped: {sorted(runtimes)}")
    P, i32, i64, u64, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64,
                            ctypes.c_size_t)
    sig = {
        "cobalt_status_string": ([ctypes.c_int], ctypes.c_char_p),
        "cobalt_layout_create": ([i32, i32, i32, i32, P, P, ctypes.POINTER(P)], ctypes.c_int),
        "cobalt_layout_destroy": ([P], ctypes.c_int),
        "cobalt_layout_tables": ([P, P, P, P], ctypes.c_int),
        "cobalt_coact_stats_workspace_bytes": ([i64, i32, i32], sz),
        "cobalt_coact_stats": ([P, i64, i32, i32, P, P, P, sz, P], ctypes.c_int),
        "cobalt_assign": ([P, P, P, i64, i32, u64, u64, i32, P, P, P], ctypes.c_int),
        "cobalt_dispatch_workspace_bytes": ([i64, i32, i32], sz),
        "cobalt_dispatch_pack": ([P, P, i64, i32, i32, P, i64, P, P, P, P, P, sz, P],
                                 ctypes.c_int),
        "cobalt_dispatch_pack_noalloc": ([P, P, i64, i32, i32, P, i64, P, P, P, P, P],
                                         ctypes.c_int),
        "cobalt_node_dispatch_workspace_bytes": ([i64, i32, i32], sz),
        "cobalt_node_dispatch_pack": ([P, P, i64, i32, i32, i32, P, i64, P, P, P, P, P, P, P, sz,
                                       P], ctypes.c_int),
        "cobalt_combine": ([P, P, P, i64, i32, i64, P, P, P], ctypes.c_int),
        "cobalt_node_combine": ([P, P, P, P, P, i64, i32, i32, i32, i64, P, P, P], ctypes.c_int),
        "cobalt_coact_ema": ([P, P, i32, ctypes.c_float, i32, P, P, P, P], ctypes.c_int),
        "cobalt_count_ema": ([P, i64, ctypes.c_float, i32, P, P], ctypes.c_int),
        "cobalt_validate_routing": ([P, P, i64, i32, i32, i32, P, P], ctypes.c_int),
        "cobalt_replica_load_workspace_bytes": ([i64, i32, i32, i32], sz),
        "cobalt_replica_load": ([P, P, i64, i32, i32, i32, P, P, sz, P], ctypes.c_int),
        "cobalt_intra_node_rebalance": ([i32, i32, i32, i32, P, P, P, P, P, P], ctypes.c_int),
        "cobalt_plan_layout": ([i32, i32, i32, i32, P, P, ctypes.c_float, P, P, P, P, P],
                               ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def _call(name: str, *args) -> None:
    st = getattr(lib(), name)(*args)
    if st != 0:
        raise CobaltError(name, st)


def _stream(stream) -> Optional[int]:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _dev(t: Optional[torch.Tensor], name: str, dtypes, shape=None) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} must have dtype in {dtypes}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t.data_ptr()


I32 = (torch.int32,)
U32 = (torch.int32, torch.uint32)  # bit patterns of uint32 counts
U16 = (torch.int16, torch.uint16)
BF16 = (torch.bfloat16,)
F32 = (torch.float32,)
I64 = (torch.int64,)
WS = (torch.uint8, torch.int8, torch.int32, torch.int64)


# ------------------------------------------------------------------- layout
class Layout:
    """Owns a cobalt_layout_t; destroyed with the object."""

    def __init__(self, handle: int, N: int, g: int, E: int, S: int):
        self.handle, self.N, self.g, self.E, self.S = handle, N, g, E, S
        self.G = N * g

    def __del__(self):
        h, self.handle = getattr(self, "handle", None), None
        if h and _lib is not None:
            _lib.cobalt_layout_destroy(h)


def cobalt_layout_create(N: int, gpus_per_node: int, E: int, S: int, slot_table,
                         owner_rank=None) -> Layout:
    st = np.ascontiguousarray(slot_table, dtype=np.int32)
    if st.shape != (N * gpus_per_node, S):
        raise ValueError(f"slot_table must be [{N * gpus_per_node}, {S}]")
    own = None if owner_rank is None else np.ascontiguousarray(owner_rank, dtype=np.int32)
    if own is not None and own.shape != (E,):
        raise ValueError(f"owner_rank must be [{E}]")
    h = ctypes.c_void_p()
    _call("cobalt_layout_create", N, gpus_per_node, E, S, st.ctypes.data_as(ctypes.c_void_p),
          None if own is None else own.ctypes.data_as(ctypes.c_void_p), ctypes.byref(h))
    return Layout(h.value, N, gpus_per_node, E, S)


def cobalt_layout_destroy(layout: Layout) -> None:
    h, layout.handle = layout.handle, None
    if h:
        _call("cobalt_layout_destroy", h)


def cobalt_layout_tables(layout: Layout):
    nm = np.zeros(layout.E, np.uint32)
    rm = np.zeros((layout.E, layout.N), np.uint32)
    own = np.zeros(layout.E, np.int32)
    _call("cobalt_layout_tables", layout.handle, nm.ctypes.data_as(ctypes.c_void_p),
          rm.ctypes.data_as(ctypes.c_void_p), own.ctypes.data_as(ctypes.c_void_p))
    return nm, rm, own


# ---------------------------------------------------------------- path calls
def cobalt_coact_stats_workspace_bytes(T: int, K: int, E: int) -> int:
    return int(lib().cobalt_coact_stats_workspace_bytes(T, K, E))


def cobalt_coact_stats(topk_idx: torch.Tensor, E: int, coact: torch.Tensor,
                       expert_count: Optional[torch.Tensor], workspace: torch.Tensor,
                       stream=None) -> None:
    T, K = topk_idx.shape
    _call("cobalt_coact_stats", _dev(topk_idx, "topk_idx", I32), T, K, E,
          _dev(coact, "coact", U32, (E, E)), _dev(expert_count, "expert_count", U32, (E,)),
          _dev(workspace, "workspace", WS), workspace.numel() * workspace.element_size(),
          _stream(stream))


def cobalt_assign(layout: Layout, topk_idx: torch.Tensor, src_rank: Optional[torch.Tensor],
                  seed: int, step: int, mode: int, assigned_rank: torch.Tensor,
                  remote_nodes: Optional[torch.Tensor] = None, stream=None) -> None:
    T, K = topk_idx.shape
    _call("cobalt_assign", layout.handle, _dev(topk_idx, "topk_idx", I32),
          _dev(src_rank, "src_rank", I32, (T,)), T, K, seed & (2**64 - 1), step & (2**64 - 1),
          mode, _dev(assigned_rank, "assigned_rank", I32, (T, K)),
          _dev(remote_nodes, "remote_nodes", U16, (T,)), _stream(stream))


def cobalt_dispatch_workspace_bytes(T: int, K: int, G: int) -> int:
    return int(lib().cobalt_dispatch_workspace_bytes(T, K, G))


def cobalt_dispatch_pack(assigned_rank: torch.Tensor, src_rank: Optional[torch.Tensor], G: int,
                         x: Optional[torch.Tensor], send_counts: torch.Tensor,
                         send_offsets: torch.Tensor, pos: torch.Tensor,
                         packed: Optional[torch.Tensor], workspace: torch.Tensor,
                         stream=None) -> None:
    T, K = assigned_rank.shape
    d = 0 if x is None else x.shape[1]
    if x is not None:
        _dev(x, "x", BF16, (T, d))
    _call("cobalt_dispatch_pack", _dev(assigned_rank, "assigned_rank", I32),
          _dev(src_rank, "src_rank", I32, (T,)), T, K, G, _dev(x, "x", BF16), d,
          _dev(send_counts, "send_counts", I32, (G, G)),
          _dev(send_offsets, "send_offsets", I64, (G * G + 1,)),
          _dev(pos, "pos", I32, (T, K)),
          _dev(packed, "packed", BF16, None if packed is None else (T * K, d)),
          _dev(workspace, "workspace", WS),
          workspace.numel() * workspace.element_size(), _stream(stream))


DISPATCH_NOALLOC_SCRATCH_BYTES = 8 << 20  # COBALT_DISPATCH_NOALLOC_SCRATCH_BYTES


def cobalt_dispatch_pack_noalloc(assigned_rank: torch.Tensor, src_rank: Optional[torch.Tensor],
                                 G: int, x: Optional[torch.Tensor], send_counts: torch.Tensor,
                                 send_offsets: torch.Tensor, pos: torch.Tensor,
                                 packed: Optional[torch.Tensor], stream=None) -> None:
    """cobalt_dispatch_pack with the library's fixed scratch in place of a
    workspace; calls that may overlap on one GPU must not be issued."""
    T, K = assigned_rank.shape
    d = 0 if x is None else x.shape[1]
    if x is not None:
        _dev(x, "x", BF16, (T, d))
    _call("cobalt_dispatch_pack_noalloc", _dev(assigned_rank, "assigned_rank", I32),
          _dev(src_rank, "src_rank", I32, (T,)), T, K, G, _dev(x, "x", BF16), d,
          _dev(send_counts, "send_counts", I32, (G, G)),
          _dev(send_offsets, "send_offsets", I64, (G * G + 1,)),
          _dev(pos, "pos", I32, (T, K)),
          _dev(packed, "packed", BF16, None if packed is None else (T * K, d)),
          _stream(stream))


def cobalt_node_dispatch_workspace_bytes(T: int, N: int, gpus_per_node: int) -> int:
    return int(lib().cobalt_node_dispatch_workspace_bytes(T, N, gpus_per_node))


def cobalt_node_dispatch_pack(assigned_rank: torch.Tensor, src_rank: Optional[torch.Tensor],
                              N: int, gpus_per_node: int, x: Optional[torch.Tensor],
                              node_counts: torch.Tensor, node_offsets: torch.Tensor,
                              node_pos: torch.Tensor, fwd_mask: torch.Tensor,
                              row_token: Optional[torch.Tensor], packed: Optional[torch.Tensor],
                              workspace: torch.Tensor, stream=None) -> None:
    """fwd_mask, row_token and packed hold T * min(K, N) rows."""
    T, K = assigned_rank.shape
    G = N * gpus_per_node
    cap = T * min(K, N)
    d = 0 if x is None else x.shape[1]
    if x is not None:
        _dev(x, "x", BF16, (T, d))
    _call("cobalt_node_dispatch_pack", _dev(assigned_rank, "assigned_rank", I32),
          _dev(src_rank, "src_rank", I32, (T,)), T, K, N, gpus_per_node, _dev(x, "x", BF16), d,
          _dev(node_counts, "node_counts", I32, (G, N)),
          _dev(node_offsets, "node_offsets", I64, (G * N + 1,)),
          _dev(node_pos, "node_pos", I32, (T, N)),
          _dev(fwd_mask, "fwd_mask", U32, (cap,)),
          _dev(row_token, "row_token", I32, (cap,)),
          _dev(packed, "packed", BF16, None if packed is None else (cap, d)),
          _dev(workspace, "workspace", WS),
          workspace.numel() * workspace.element_size(), _stream(stream))


EMA_INIT, EMA_CLEAR = 1, 2


def cobalt_coact_ema(coact: torch.Tensor, expert_count: torch.Tensor, decay: float,
                     flags: int = 0, ema_coact: Optional[torch.Tensor] = None,
                     ema_count: Optional[torch.Tensor] = None,
                     ochiai: Optional[torch.Tensor] = None, stream=None) -> None:
    E = expert_count.shape[0]
    _call("cobalt_coact_ema", _dev(coact, "coact", U32, (E, E)),
          _dev(expert_count, "expert_count", U32, (E,)), E, float(decay), int(flags),
          _dev(ema_coact, "ema_coact", F32, (E, E)), _dev(ema_count, "ema_count", F32, (E,)),
          _dev(ochiai, "ochiai", F32, (E, E)), _stream(stream))


def cobalt_count_ema(counts: torch.Tensor, decay: float, flags: int = 0,
                     ema: Optional[torch.Tensor] = None, stream=None) -> None:
    n = counts.numel()
    _call("cobalt_count_ema", _dev(counts, "counts", U32), n, float(decay), int(flags),
          _dev(ema, "ema", F32, tuple(counts.shape)), _stream(stream))


def cobalt_combine(expert_out: torch.Tensor, pos: torch.Tensor, gates: torch.Tensor,
                   y: torch.Tensor, y_f32: Optional[torch.Tensor] = None, stream=None) -> None:
    T, K = pos.shape
    d = y.shape[1]
    _call("cobalt_combine", _dev(expert_out, "expert_out", BF16, (T * K, d)),
          _dev(pos, "pos", I32), _dev(gates, "gates", F32, (T, K)), T, K, d,
          _dev(y, "y", BF16, (T, d)), _dev(y_f32, "y_f32", F32, (T, d)), _stream(stream))


def cobalt_node_combine(expert_out: torch.Tensor, pos: torch.Tensor, assigned_rank: torch.Tensor,
                        gates: torch.Tensor, node_pos: torch.Tensor, N: int, gpus_per_node: int,
                        node_partial: torch.Tensor, y: torch.Tensor, stream=None) -> None:
    """node_partial holds T * min(K, N) rows; node_pos comes from
    cobalt_node_dispatch_pack on the same assigned ranks."""
    T, K = pos.shape
    d = y.shape[1]
    _call("cobalt_node_combine", _dev(expert_out, "expert_out", BF16, (T * K, d)),
          _dev(pos, "pos", I32, (T, K)), _dev(assigned_rank, "assigned_rank", I32, (T, K)),
          _dev(gates, "gates", F32, (T, K)), _dev(node_pos, "node_pos", I32, (T, N)), T, K, N,
          gpus_per_node, d, _dev(node_partial, "node_partial", BF16, (T * min(K, N), d)),
          _dev(y, "y", BF16, (T, d)), _stream(stream))


def cobalt_replica_load_workspace_bytes(T: int, K: int, E: int, G: int) -> int:
    return int(lib().cobalt_replica_load_workspace_bytes(T, K, E, G))


def cobalt_replica_load(topk_idx: torch.Tensor, assigned_rank: torch.Tensor, E: int, G: int,
                        load: torch.Tensor, workspace: torch.Tensor, stream=None) -> None:
    T, K = topk_idx.shape
    _call("cobalt_replica_load", _dev(topk_idx, "topk_idx", I32),
          _dev(assigned_rank, "assigned_rank", I32, (T, K)), T, K, E, G,
          _dev(load, "load", U32, (E, G)), _dev(workspace, "workspace", WS),
          workspace.numel() * workspace.element_size(), _stream(stream))


def cobalt_intra_node_rebalance(N: int, gpus_per_node: int, E: int, S: int, slot_table,
                                owner_rank, replica_load):
    """Host-only Stage-2 rebalancing. Returns (new_slot_table [G, S] int32,
    new_owner_rank [E] int32, rank_load [G] float32)."""
    G = N * gpus_per_node
    st = np.ascontiguousarray(slot_table, dtype=np.int32)
    if st.shape != (G, S):
        raise ValueError(f"slot_table must be [{G}, {S}]")
    own = None if owner_rank is None else np.ascontiguousarray(owner_rank, dtype=np.int32)
    rl = np.ascontiguousarray(replica_load, dtype=np.float32)
    if rl.shape != (E, G):
        raise ValueError(f"replica_load must be [{E}, {G}]")
    out = np.zeros((G, S), np.int32)
    new_own = np.zeros(E, np.int32)
    rank_load = np.zeros(G, np.float32)
    P = ctypes.c_void_p
    _call("cobalt_intra_node_rebalance", N, gpus_per_node, E, S, st.ctypes.data_as(P),
          None if own is None else own.ctypes.data_as(P), rl.ctypes.data_as(P),
          out.ctypes.data_as(P), new_own.ctypes.data_as(P), rank_load.ctypes.data_as(P))
    return out, new_own, rank_load


def cobalt_plan_layout(N: int, gpus_per_node: int, E: int, S: int, coact_ema, count_ema,
                       eps: float = 0.15):
    """Host-only Stage-1 planner. Returns (slot_table [G, S] int32,
    owner_rank [E] int32, plan [E, G] float32, objective float, feasible
    bool). coact_ema [E, E] and count_ema [E] are host arrays or tensors."""
    G = N * gpus_per_node
    if isinstance(coact_ema, torch.Tensor):
        coact_ema = coact_ema.detach().cpu().numpy()
    if isinstance(count_ema, torch.Tensor):
        count_ema = count_ema.detach().cpu().numpy()
    c = np.ascontiguousarray(coact_ema, dtype=np.float32)
    w = np.ascontiguousarray(count_ema, dtype=np.float32)
    if c.shape != (E, E) or w.shape != (E,):
        raise ValueError(f"coact_ema must be [{E}, {E}] and count_ema [{E}]")
    table = np.zeros((G, S), np.int32)
    owner = np.zeros(E, np.int32)
    plan = np.zeros((E, G), np.float32)
    obj = ctypes.c_double()
    feas = ctypes.c_int32()
    P = ctypes.c_void_p
    _call("cobalt_plan_layout", N, gpus_per_node, E, S, c.ctypes.data_as(P), w.ctypes.data_as(P),
          float(eps), table.ctypes.data_as(P), owner.ctypes.data_as(P), plan.ctypes.data_as(P),
          ctypes.byref(obj), ctypes.byref(feas))
    return table, owner, plan, obj.value, bool(feas.value)


def replica_load_workspace_for(T: int, K: int, E: int, G: int, device="cuda") -> torch.Tensor:
    n = cobalt_replica_load_workspace_bytes(T, K, E, G)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


def cobalt_validate_routing(topk_idx: torch.Tensor, src_rank: Optional[torch.Tensor], E: int,
                            G: int, stream=None) -> int:
    """Returns the violation bitmask (0 = valid); see include/cobalt.h."""
    T, K = topk_idx.shape
    flags = ctypes.c_uint32(0)
    st = lib().cobalt_validate_routing(_dev(topk_idx, "topk_idx", I32),
                                       _dev(src_rank, "src_rank", I32, (T,)), T, K, E, G,
                                       ctypes.byref(flags), _stream(stream))
    if st not in (0, 5):
        raise CobaltError("cobalt_validate_routing", st)
    return int(flags.value)


def workspace_for(T: int, K: int, G: int, device="cuda") -> torch.Tensor:
    """A dispatch workspace of the size the library asks for."""
    n = cobalt_dispatch_workspace_bytes(T, K, G)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


def node_workspace_for(T: int, N: int, gpus_per_node: int, device="cuda") -> torch.Tensor:
    """A node-deduplicated dispatch workspace of the size the library asks for."""
    n = cobalt_node_dispatch_workspace_bytes(T, N, gpus_per_node)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


def stats_workspace_for(T: int, K: int, E: int, device="cuda") -> torch.Tensor:
    """A statistics workspace of the size the library asks for."""
    n = cobalt_coact_stats_workspace_bytes(T, K, E)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)
