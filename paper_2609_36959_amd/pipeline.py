"""One routing step on the GPU: device buffers for a workload and the four
library calls in stream order (statistics, assignment, dispatch/pack,
combine). Used by the benchmark, the smoke check and the full-size tests so
that all of them run the same launches."""
from __future__ import annotations

from typing import Optional

import numpy as np
import torch

from . import binding as B
from . import workload as W


class RoutingStep:
    """Device state of one workload.

    expert_out: "independent" draws a separate bf16 buffer in packed layout
    (a stand-in for the experts' outputs); "roundtrip" feeds the packed rows
    back, so the combine must return x when the gates sum to one.
    """

    def __init__(self, w: W.Workload, seed: int, device="cuda", expert_out="independent",
                 src: Optional[np.ndarray] = None, step: int = 0, layout=None,
                 route_device: Optional[str] = None):
        self.w, self.seed, self.device = w, seed, torch.device(device)
        dev = self.device
        T, K, E, G, d = w.T, w.K, w.E, w.G, w.d
        rd = route_device if route_device is not None else device
        self.src_np = src
        self.src = None if src is None else torch.from_numpy(np.ascontiguousarray(src, np.int32)).to(dev)
        table, owner = layout if layout is not None else W.layout(w, seed)
        self.table, self.owner = table, owner
        self.layout = B.cobalt_layout_create(w.N, w.g, E, table.shape[1], table, owner)
        self.set_routing(step, rd)
        self.x = W.hidden(w, seed, device=dev)
        self.coact = torch.zeros(E, E, dtype=torch.int32, device=dev)
        self.count = torch.zeros(E, dtype=torch.int32, device=dev)
        self.assigned = torch.empty(T, K, dtype=torch.int32, device=dev)
        self.remote = torch.empty(T, dtype=torch.int16, device=dev)
        self.counts = torch.empty(G, G, dtype=torch.int32, device=dev)
        self.offsets = torch.empty(G * G + 1, dtype=torch.int64, device=dev)
        self.pos = torch.empty(T, K, dtype=torch.int32, device=dev)
        self.packed = torch.empty(T * K, d, dtype=torch.bfloat16, device=dev)
        self.expert_mode = expert_out
        if expert_out == "independent":
            self.eo = W.expert_outputs(w, seed, device=dev)
        elif expert_out == "roundtrip":
            self.eo = self.packed
        else:
            raise ValueError(expert_out)
        self.y = torch.empty(T, d, dtype=torch.bfloat16, device=dev)
        self.workspace = B.workspace_for(T, K, G, device=dev)
        self.stats_workspace = B.stats_workspace_for(T, K, E, device=dev)
        self.replica_load = torch.zeros(E, G, dtype=torch.int32, device=dev)
        self.load_workspace = B.replica_load_workspace_for(T, K, E, G, device=dev)

    def set_routing(self, step: int, route_device=None):
        rd = self.device if route_device is None else route_device
        topk, gates = W.routing(self.w, self.seed, step=step, device=rd)
        self.topk = topk.to(self.device).contiguous()
        self.gates = gates.to(self.device).contiguous()
        self.step = step

    def set_layout(self, table, owner):
        self.table, self.owner = table, owner
        B.cobalt_layout_destroy(self.layout)
        self.layout = B.cobalt_layout_create(self.w.N, self.w.g, self.w.E, table.shape[1],
                                             table, owner)

    # the four calls of one step ------------------------------------------
    def stats(self, stream=None):
        B.cobalt_coact_stats(self.topk, self.w.E, self.coact, self.count, self.stats_workspace,
                             stream=stream)

    def assign(self, mode=0, stream=None):
        B.cobalt_assign(self.layout, self.topk, self.src, self.seed, self.step, mode,
                        self.assigned, self.remote, stream=stream)

    def pack(self, stream=None):
        B.cobalt_dispatch_pack(self.assigned, self.src, self.w.G, self.x, self.counts,
                               self.offsets, self.pos, self.packed, self.workspace, stream=stream)

    def combine(self, y_f32=None, stream=None):
        B.cobalt_combine(self.eo, self.pos, self.gates, self.y, y_f32, stream=stream)

    def load(self, stream=None):
        """Adds this step's per-replica task counts w_er into replica_load."""
        B.cobalt_replica_load(self.topk, self.assigned, self.w.E, self.w.G, self.replica_load,
                              self.load_workspace, stream=stream)

    def node_pack(self, stream=None):
        """Node-deduplicated dispatch layout and pack of the current
        assignment (one row per (token, destination node)); buffers are
        allocated on first use."""
        w = self.w
        if getattr(self, "node_packed", None) is None:
            dev, cap = self.device, w.T * min(w.K, w.N)
            self.node_counts = torch.empty(w.G, w.N, dtype=torch.int32, device=dev)
            self.node_offsets = torch.empty(w.G * w.N + 1, dtype=torch.int64, device=dev)
            self.node_pos = torch.empty(w.T, w.N, dtype=torch.int32, device=dev)
            self.fwd_mask = torch.empty(cap, dtype=torch.int32, device=dev)
            self.row_token = torch.empty(cap, dtype=torch.int32, device=dev)
            self.node_packed = torch.empty(cap, w.d, dtype=torch.bfloat16, device=dev)
            self.node_workspace = B.node_workspace_for(w.T, w.N, w.g, device=dev)
        B.cobalt_node_dispatch_pack(self.assigned, self.src, w.N, w.g, self.x, self.node_counts,
                                    self.node_offsets, self.node_pos, self.fwd_mask,
                                    self.row_token, self.node_packed, self.node_workspace,
                                    stream=stream)

    def node_combine(self, stream=None):
        """Node-level combine of the expert outputs over the node rows of the
        last node_pack: bf16 partials per (token, node) in node_partial, then
        y_node; buffers are allocated on first use."""
        w = self.w
        if getattr(self, "node_partial", None) is None:
            cap = w.T * min(w.K, w.N)
            self.node_partial = torch.empty(cap, w.d, dtype=torch.bfloat16, device=self.device)
            self.y_node = torch.empty(w.T, w.d, dtype=torch.bfloat16, device=self.device)
        B.cobalt_node_combine(self.eo, self.pos, self.assigned, self.gates, self.node_pos, w.N,
                              w.g, self.node_partial, self.y_node, stream=stream)

    def ema(self, decay: float, flags: int = 0, stream=None):
        """Folds the accumulated counts into the planner EMAs (ema_coact,
        ema_count) and writes the Ochiai similarity of the counts; buffers are
        allocated on first use. flags: B.EMA_INIT, B.EMA_CLEAR."""
        if getattr(self, "ochiai", None) is None:
            E, dev = self.w.E, self.device
            self.ema_coact = torch.zeros(E, E, dtype=torch.float32, device=dev)
            self.ema_count = torch.zeros(E, dtype=torch.float32, device=dev)
            self.ochiai = torch.zeros(E, E, dtype=torch.float32, device=dev)
        B.cobalt_coact_ema(self.coact, self.count, decay, flags, self.ema_coact, self.ema_count,
                           self.ochiai, stream=stream)

    def run(self, mode=0, stream=None):
        self.stats(stream)
        self.assign(mode, stream)
        self.pack(stream)
        self.combine(stream=stream)

    def close(self):
        if self.layout is not None:
            B.cobalt_layout_destroy(self.layout)
            self.layout = None


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Raw bf16 bit patterns of a tensor as uint16 (host copy)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
