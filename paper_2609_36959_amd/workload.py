"""Seeded synthetic workloads for the co-activation routing path.

This module only draws inputs: per-token expert selections and gates, hidden
states, stand-in expert outputs, source ranks, and an expert layout (the
replica table a host planner would hand over). It computes none of the
routing path's steps; both the HIP library and the oracle consume what it
returns.

Shapes follow the problem statement of the Cobalt paper (Section 3.1,
notation table): T tokens, E experts, top-K selections per token, G = N*g
ranks on N nodes, S replica slots per rank (S = (1+rho)E/G, Section 3.1).

Routing recipe (stands in for gating on C4 with the paper's models, whose
traces are not available):
  logits[t, e] = z[t, e] + bias[e] + beta * [e in cluster(c_t)]
  z ~ N(0, 1) fp32; bias[e] = -alpha * ln(pi(e) + 1) with pi a seeded
  permutation (a log-Zipf popularity skew); clusters are a seeded partition
  of the experts into groups of `cluster_size`, each token picks one cluster
  uniformly (planted co-activation). Slot j of topk_idx is the j-th largest
  logit; gates are a softmax over the K selected logits in fp32.

The routing arrays are drawn with torch's generator on the requested device;
the stream therefore depends on the device type (CPU and GPU draws differ),
and every consumer is handed the same arrays.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Sequence

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    T: int                 # tokens per step
    E: int                 # experts
    K: int                 # experts per token
    d: int                 # hidden size (bf16 elements per row)
    N: int                 # nodes
    g: int                 # GPUs (ranks) per node
    S: int                 # replica slots per rank
    zipf_alpha: float = 0.0
    cluster_size: int = 0
    cluster_beta: float = 0.0
    owners: str = "contiguous"      # "permuted" | "contiguous" | "cluster"
    replicas: str = "random"        # "random" | "intra_node_top"
    top_frac: float = 0.10          # replicated share for "intra_node_top"
    steps: int = 1
    drift_frac: float = 0.0         # share of experts whose bias rotates per step
    swap_step: int = -1             # step before which the layout is re-planned
    seed: int = 0                   # default seed of the workload

    @property
    def G(self) -> int:
        return self.N * self.g

    def describe(self) -> str:
        return (f"T={self.T} E={self.E} K={self.K} d={self.d} "
                f"{self.N}x{self.g} S={self.S}")


# The five seeded workloads, by name. The tiny workload's slot count reads
# "2 slots (owner + 1 replica)" with E/G = 2 owners per rank, which leaves no
# room for a replica; it is read as 3 slots (rho = 0.5), and the literal 2 is
# kept as the no-replica degenerate case in the tests.
WORKLOADS = {w.name: w for w in (
    Workload("tiny", 4096, 16, 2, 512, 2, 4, 3, zipf_alpha=1.0,
             owners="permuted", replicas="random", seed=0),
    Workload("clusters-e64", 16384, 64, 6, 2048, 4, 8, 3,
             cluster_size=4, cluster_beta=2.0,
             owners="contiguous", replicas="random", seed=1),
    Workload("colocate-e128", 65536, 128, 8, 4096, 4, 8, 5, zipf_alpha=1.2,
             cluster_size=8, cluster_beta=1.5,
             owners="cluster", replicas="intra_node_top", seed=2),
    Workload("colocate-e256", 131072, 256, 8, 7168, 8, 8, 5, zipf_alpha=1.1,
             cluster_size=4, cluster_beta=2.0,
             owners="cluster", replicas="intra_node_top", seed=3),
    Workload("drift-e384", 262144, 384, 8, 7168, 8, 8, 8, zipf_alpha=1.1,
             owners="contiguous", replicas="random",
             steps=16, drift_frac=0.05, swap_step=8, seed=4),
)}
NAMES = list(WORKLOADS)

# numbered sub-streams of a seed
_S_PERM, _S_CLUSTER, _S_LAYOUT, _S_DRIFT, _S_ROUTE, _S_HIDDEN, _S_EXPOUT, _S_HOT = range(8)


def _np_rng(seed: int, stream: int, *extra: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream, *extra])))


def _torch_seed(seed: int, stream: int, *extra: int) -> int:
    return int(np.random.SeedSequence([seed, stream, *extra]).generate_state(1, np.uint64)[0] >> 1)


def with_sizes(w: Workload, **kw) -> Workload:
    """Same recipe at other sizes (used for reduced-T test cases)."""
    return dataclasses.replace(w, **kw)


# --------------------------------------------------------------------------
# expert popularity and clusters
# --------------------------------------------------------------------------
def zipf_rank(w: Workload, seed: int) -> np.ndarray:
    """pi(e): the popularity rank of expert e (0 = most popular)."""
    return _np_rng(seed, _S_PERM).permutation(w.E).astype(np.int64)


def bias(w: Workload, seed: int, step: int = 0) -> np.ndarray:
    """Per-expert logit bias at `step` (fp32). With drift, each step rotates
    the bias values of round(drift_frac * E) seeded experts by one place."""
    if w.zipf_alpha > 0:
        b = (-w.zipf_alpha * np.log(zipf_rank(w, seed).astype(np.float64) + 1.0))
    else:
        b = np.zeros(w.E)
    if w.drift_frac > 0:
        m = int(round(w.drift_frac * w.E))
        for s in range(1, step + 1):
            sel = _np_rng(seed, _S_DRIFT, s).choice(w.E, size=m, replace=False)
            b[sel] = np.roll(b[sel], 1)
    return b.astype(np.float32)


def clusters(w: Workload, seed: int) -> Optional[np.ndarray]:
    """[E/cluster_size, cluster_size] expert ids per cluster, or None."""
    if w.cluster_size <= 0:
        return None
    perm = _np_rng(seed, _S_CLUSTER).permutation(w.E)
    return perm.reshape(w.E // w.cluster_size, w.cluster_size).astype(np.int64)


def expected_hot_order(w: Workload, seed: int) -> np.ndarray:
    """Experts from most to least popular in expectation under the routing
    recipe. Cluster boosts are uniform over clusters, so the order is the
    Zipf rank; without a Zipf skew every expert is equally popular and a
    seeded permutation decides."""
    if w.zipf_alpha > 0:
        return np.argsort(zipf_rank(w, seed), kind="stable").astype(np.int64)
    return _np_rng(seed, _S_HOT).permutation(w.E).astype(np.int64)


# --------------------------------------------------------------------------
# routing: topk_idx [T, K] int32, gates [T, K] fp32
# --------------------------------------------------------------------------
def routing(w: Workload, seed: int, step: int = 0, device="cpu",
            chunk: int = 1 << 16):
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(_torch_seed(seed, _S_ROUTE, step))
    b = torch.from_numpy(bias(w, seed, step)).to(dev)
    cl = clusters(w, seed)
    cl_t = torch.from_numpy(cl).to(dev) if cl is not None else None
    idx_out = torch.empty(w.T, w.K, dtype=torch.int32, device=dev)
    gate_out = torch.empty(w.T, w.K, dtype=torch.float32, device=dev)
    for t0 in range(0, w.T, chunk):
        n = min(chunk, w.T - t0)
        logits = torch.randn(n, w.E, generator=gen, device=dev, dtype=torch.float32)
        logits += b
        if cl_t is not None:
            c = torch.randint(cl_t.shape[0], (n,), generator=gen, device=dev)
            boost = torch.full((n, w.cluster_size), w.cluster_beta, device=dev)
            logits.scatter_add_(1, cl_t[c], boost)
        vals, idx = torch.topk(logits, w.K, dim=1, largest=True, sorted=True)
        idx_out[t0:t0 + n] = idx.to(torch.int32)
        gate_out[t0:t0 + n] = torch.softmax(vals, dim=1)
    return idx_out, gate_out


def contiguous_src(T: int, G: int) -> np.ndarray:
    """Source rank of each token when the T tokens are split into G equal
    contiguous blocks (what the library assumes for a NULL src_rank)."""
    assert T % G == 0
    return (np.arange(T, dtype=np.int64) // (T // G)).astype(np.int32)


def ragged_src(T: int, G: int, seed: int) -> np.ndarray:
    """Non-decreasing source ranks with uneven block sizes (some empty)."""
    r = _np_rng(seed, _S_LAYOUT, 99)
    cuts = np.sort(r.integers(0, T + 1, size=G - 1))
    return np.searchsorted(cuts, np.arange(T), side="right").astype(np.int32)


# --------------------------------------------------------------------------
# hidden states and stand-in expert outputs (bf16, returned as torch tensors)
# --------------------------------------------------------------------------
def _normal_bf16(rows: int, d: int, seed: int, device, chunk_elems: int = 1 << 26):
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    out = torch.empty(rows, d, dtype=torch.bfloat16, device=dev)
    step = max(1, chunk_elems // max(d, 1))
    for r0 in range(0, rows, step):
        n = min(step, rows - r0)
        out[r0:r0 + n] = torch.randn(n, d, generator=gen, device=dev,
                                     dtype=torch.float32).to(torch.bfloat16)
    return out


def hidden(w: Workload, seed: int, device="cpu", step: int = 0, T: Optional[int] = None):
    """x [T, d] bf16 ~ N(0, 1)."""
    return _normal_bf16(T if T is not None else w.T, w.d,
                        _torch_seed(seed, _S_HIDDEN, step), device)


def expert_outputs(w: Workload, seed: int, device="cpu", step: int = 0,
                   rows: Optional[int] = None):
    """Stand-in expert outputs [T*K, d] bf16 ~ N(0, 1) in packed-row order."""
    return _normal_bf16(rows if rows is not None else w.T * w.K, w.d,
                        _torch_seed(seed, _S_EXPOUT, step), device)


# --------------------------------------------------------------------------
# expert layout (the planner's output, here drawn from a recipe)
# --------------------------------------------------------------------------
def layout(w: Workload, seed: int, hot_order: Optional[Sequence[int]] = None,
           S: Optional[int] = None, replicas: Optional[str] = None,
           owners: Optional[str] = None, plan: int = 0):
    """Return (slot_table [G, S] int32 with -1 = empty, owner_rank [E] int32).

    owners:
      "permuted"   a seeded permutation of experts dealt E/G per rank
      "contiguous" expert e on rank e // (E/G)
      "cluster"    cluster c goes to node order[c] (round-robin over nodes in
                   a seeded order), its members dealt round-robin to that
                   node's ranks (co-location of planted clusters)
    replicas:
      "none"           owners only
      "random"         the G*S - E hottest experts get one replica each, on a
                       uniformly drawn rank with a free slot that does not
                       already hold the expert
      "intra_node_top" the round(top_frac * E) hottest experts get one replica
                       each on the owner's node: the least-filled other rank
                       of that node with a free slot (lowest id on ties)
    `hot_order` lists experts from hottest down; default is the expected
    popularity under the routing recipe. `plan` numbers re-plans of the
    same workload (it reseeds the random placement).
    """
    S = w.S if S is None else S
    replicas = w.replicas if replicas is None else replicas
    owners = w.owners if owners is None else owners
    E, G, N, g = w.E, w.G, w.N, w.g
    assert E % G == 0, "owners are dealt E/G per rank"
    per = E // G
    assert S >= per
    r = _np_rng(seed, _S_LAYOUT, plan)
    owner = np.empty(E, dtype=np.int64)
    if owners == "contiguous":
        owner[:] = np.arange(E) // per
    elif owners == "permuted":
        owner[r.permutation(E)] = np.arange(E) // per
    elif owners == "cluster":
        cl = clusters(w, seed)
        assert cl is not None and cl.shape[0] % N == 0
        node_order = r.permutation(N)
        fill = np.zeros(N, dtype=np.int64)
        for c in range(cl.shape[0]):
            n = node_order[c % N]
            for e in cl[c]:
                owner[e] = n * g + (fill[n] % g)
                fill[n] += 1
        assert np.all(np.bincount(owner, minlength=G) == per)
    else:
        raise ValueError(owners)

    slots = [[int(e) for e in np.flatnonzero(owner == rk)] for rk in range(G)]
    hot = np.asarray(expected_hot_order(w, seed) if hot_order is None else hot_order,
                     dtype=np.int64)

    if replicas == "random":
        for e in hot[: G * S - E]:
            cand = [rk for rk in range(G) if len(slots[rk]) < S and e not in slots[rk]]
            if not cand:
                continue  # the only free slots are on ranks already holding e
            slots[cand[int(r.integers(len(cand)))]].append(int(e))
    elif replicas == "intra_node_top":
        for e in hot[: int(round(w.top_frac * E))]:
            n = owner[e] // g
            cand = [rk for rk in range(n * g, (n + 1) * g)
                    if len(slots[rk]) < S and e not in slots[rk]]
            if not cand:
                continue
            best = min(cand, key=lambda rk: (len(slots[rk]), rk))
            slots[best].append(int(e))
    elif replicas != "none":
        raise ValueError(replicas)

    table = np.full((G, S), -1, dtype=np.int32)
    for rk in range(G):
        table[rk, : len(slots[rk])] = slots[rk]
    return table, owner.astype(np.int32)


def contiguous_ep_layout(w: Workload):
    """Plain expert parallelism: contiguous owners, no replicas."""
    return layout(w, 0, S=w.E // w.G, replicas="none", owners="contiguous")
