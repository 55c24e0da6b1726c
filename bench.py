"""Benchmark of the co-activation routing path on one MI355X.

One step = one pass of the whole path over one batch: co-activation
statistics, communication-aware assignment (Algorithm 1), dispatch layout +
pack, and the gate-weighted combine, on the workload with T=131072 tokens,
E=256 experts, top-8, d=7168 bf16, 8 virtual nodes x 8 GPUs, 5 slots per
GPU (co-located planted clusters, Zipf-skewed popularity). Inputs are
seeded synthetic data resident in HBM before timing starts.

Prints one JSON line: routed tokens/s over the timed steps, the roofline
position of the dominant call, the pack+combine share of HBM peak, routing
quality (cross-node traffic of Algorithm 1 vs owner-only baselines), and the
oracle's CPU throughput on a bounded sample of the same workload.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12  # MI355X HBM3E, bytes/s
METRIC = "routed tokens/sec (stats+assign+pack+combine), % of HBM peak, 1 MI355X"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_{call}_{workload}.txt")
KERNEL_SOURCES = {"cobalt_dispatch_pack": "dispatch.hip", "cobalt_combine": "combine.hip",
                  "cobalt_node_dispatch_pack": "dispatch.hip", "cobalt_node_combine": "combine.hip"}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="colocate-e256",
                    help="name of a seeded workload in paper_2609_36959_amd/workload.py")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-tokens", type=int, default=65536)
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the extra timing of the step replayed as a HIP graph")
    ap.add_argument("--headline-only", action="store_true",
                    help="time only the named workload (no per-workload summaries)")
    ap.add_argument("--workloads", default="all",
                    help="comma-separated workloads to summarise beside the named one "
                         "(default: all five)")
    ap.add_argument("--replan", choices=("planner", "recipe"), default="planner",
                    help="multi-step workloads: re-plan the layout with the Stage-1 planner "
                         "from the EMA statistics, or with the workload's hot-order recipe")
    return ap.parse_args()


def algorithmic_bytes(w):
    """Bytes each call must move (read + write), per call (one step)."""
    T, K, d, E, G = w.T, w.K, w.d, w.E, w.G
    return {
        "cobalt_coact_stats": T * K * 4 + 2 * 4 * (E * E + E),
        # counts read and cleared, EMA read and written, Ochiai written
        "cobalt_coact_ema": E * E * 4 * 5 + E * 4 * 4,
        "cobalt_assign": T * K * 4 + T * K * 4 + T * 2,
        "cobalt_dispatch_pack": T * d * 2 + T * K * d * 2 + T * K * 8 + 12 * G * G,
        "cobalt_combine": T * K * d * 2 + T * K * 8 + T * d * 2,
    }


def node_dispatch_bytes(w, rows):
    """Bytes the node-deduplicated dispatch must move for `rows` node rows:
    read the assignment and x once, write the packed rows, node_pos, the
    forwarding masks and row tokens, and the [G][N] counts and offsets."""
    T, K, d, N, G = w.T, w.K, w.d, w.N, w.G
    return T * K * 4 + T * d * 2 + rows * d * 2 + T * N * 4 + rows * 8 + 12 * G * N


def node_combine_bytes(w, rows):
    """Bytes the node-level combine must move: the node side reads every
    pair's expert row, its pos, rank and gate and the node rows, and writes
    `rows` bf16 partials; the source side reads the partials and node_pos
    and writes y."""
    T, K, d, N = w.T, w.K, w.d, w.N
    return T * K * d * 2 + T * K * 12 + 2 * T * N * 4 + 2 * rows * d * 2 + T * d * 2


def source_digest(call):
    p = os.path.join(ROOT, "paper_2609_36959_amd", "csrc", KERNEL_SOURCES[call])
    return hashlib.sha256(open(p, "rb").read()).hexdigest()[:16]


def measured_traffic(call, workload):
    """HBM bytes per call from committed rocprofv3 counter runs, if they were
    taken on the current kernel source; else None."""
    p = TRAFFIC_FILE.format(call=call, workload=workload)
    if not os.path.exists(p):
        return None
    kv = {}
    for line in open(p):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256_16") != source_digest(call):
        return None
    try:
        return float(kv["hbm_bytes_per_call"])
    except (KeyError, ValueError):
        return None


class RoutingTally:
    """Cross-node traffic (Eq. 1) of Algorithm 1 against two owner-only
    baselines, summed over the steps added: owner-only on the same layout,
    and owner-only on plain contiguous expert parallelism without replicas.
    Sources are the contiguous blocks of the step. Reporting only (outside
    the timed region)."""

    def __init__(self, w, seed, torch, B, W):
        self.w, self.seed, self.torch, self.B = w, seed, torch, B
        t, o = W.contiguous_ep_layout(w)
        self.ep = B.cobalt_layout_create(w.N, w.g, w.E, t.shape[1], t, o)
        self.acc = {k: [0, 0, 0.0] for k in ("alg1", "owner_only", "contiguous_ep_owner_only")}
        self.per_step_V = []
        self.steps = 0

    def _measure(self, layout, topk, step, mode):
        torch, w = self.torch, self.w
        a = torch.empty(w.T, w.K, dtype=torch.int32, device=topk.device)
        rn = torch.empty(w.T, dtype=torch.int16, device=topk.device)
        self.B.cobalt_assign(layout, topk, None, self.seed, step, mode, a, rn)
        torch.cuda.synchronize()
        src_node = (torch.arange(w.T, device=a.device) // (w.T // w.G)) // w.g
        cross = (a // w.g != src_node[:, None]).sum().item()
        rn32 = rn.to(torch.int32) & 0xFFFF
        V = sum(((rn32 >> n) & 1).sum().item() for n in range(w.N))
        load = torch.bincount(a.flatten(), minlength=w.G).float()
        return int(V), int(cross), float(load.max() / load.mean())

    def add(self, layout, topk, step):
        for key, L, mode in (("alg1", layout, 0), ("owner_only", layout, 1),
                             ("contiguous_ep_owner_only", self.ep, 1)):
            V, cross, imb = self._measure(L, topk, step, mode)
            a = self.acc[key]
            a[0] += V
            a[1] += cross
            a[2] += imb
            if key == "alg1":
                self.per_step_V.append(V)
        self.steps += 1

    def report(self):
        w, n = self.w, max(self.steps, 1)
        out = {k: {"V": a[0], "cross_pair_frac": a[1] / (n * w.T * w.K), "imbalance": a[2] / n}
               for k, a in self.acc.items()}
        for k in ("owner_only", "contiguous_ep_owner_only"):
            base = out[k]["V"]
            out[f"V_reduction_vs_{k}"] = 1.0 - out["alg1"]["V"] / base if base else 0.0
        if self.steps > 1:
            out["steps_summed"] = self.steps
            out["alg1_V_per_step"] = self.per_step_V
        return out

    def close(self):
        if self.ep is not None:
            self.B.cobalt_layout_destroy(self.ep)
            self.ep = None


def routing_quality(st, torch, B, W):
    """RoutingTally of the current step on the current layout."""
    t = RoutingTally(st.w, st.seed, torch, B, W)
    try:
        t.add(st.layout, st.topk, 0)
        return t.report()
    finally:
        t.close()


def device_info(torch):
    """hipDeviceProp of device 0, as torch reports it."""
    p = torch.cuda.get_device_properties(0)
    out = {"name": p.name, "compute_units": p.multi_processor_count,
           "hbm_bytes": p.total_memory}
    for k in ("gcnArchName", "L2_cache_size"):
        if hasattr(p, k):
            out[k] = getattr(p, k)
    return out


def hbm_reference(torch, stream, st, reps=5):
    """HBM rates measured live on this device, on the bench's stream, with
    the reference kernels of paper_2609_36959_amd/ceilings (each checked by
    tests/test_gpu_ceilings.py to move the bytes it counts):
    - read, write_fill, copy: one-pass streaming kernels on 4 GiB buffers
      (16 B non-temporal accesses, one per thread), and torch's fill beside
      them;
    - pack_store: the pack's own store pattern on this step's pos (one
      workgroup per token and 2 KiB slice, a 2 KiB burst per slot) without
      its loads of x, the ceiling of the pack's write shape;
    - gather_read: the combine's own loads of the K packed rows per token
      and slice without the fold and the stores of y, the floor of its read
      shape."""
    from paper_2609_36959_amd import ceilings as CL
    n = 1 << 30  # int32 elements: 4 GiB
    a = torch.ones(n, dtype=torch.int32, device="cuda")
    b = torch.empty_like(a)
    xo = torch.empty(CL.stream_blocks(4 * n), dtype=torch.int32, device="cuda")
    w = st.w
    groups = (w.d // 8 + 127) // 128
    go = torch.empty(w.T * groups, dtype=torch.int32, device="cuda")
    pk = w.T * w.K * w.d * 2
    out = {}
    with torch.cuda.stream(stream):
        for name, fn, nbytes in (
                ("read", lambda: CL.read(a, xo, stream=stream), 4 * n),
                ("write_fill", lambda: CL.fill(b, stream=stream), 4 * n),
                ("copy", lambda: CL.copy(a, b, stream=stream), 8 * n),
                ("torch_fill", lambda: b.fill_(3), 4 * n),
                ("pack_store", lambda: CL.pack_store(st.pos, st.packed, stream=stream), pk),
                ("gather_read", lambda: CL.gather_read(st.eo, st.pos, go, stream=stream), pk)):
            fn()
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            ev[0].record(stream)
            for _ in range(reps):
                fn()
            ev[1].record(stream)
            torch.cuda.synchronize()
            ms = ev[0].elapsed_time(ev[1]) / reps
            out[name] = {"GB_s": round(nbytes / (ms * 1e-3) / 1e9, 1), "ms": round(ms, 4)}
    del a, b
    torch.cuda.empty_cache()
    # the pack's rows are rewritten by the step's own pack
    with torch.cuda.stream(stream):
        st.pack(stream=stream)
    torch.cuda.synchronize()
    return out | {"buffer": "4 GiB for the streaming kernels; this step's pos, packed rows and "
                            "expert outputs for pack_store and gather_read"}


def stage2_demo(st, torch, B, W):
    """Per-step intra-node rebalancing (Section 3.2, Stage 2) on this step:
    the per-replica loads w_er measured on the GPU drive the host greedy
    re-placement; the step is then re-assigned on the new layout. Reports
    the rank-load imbalance (max / mean) before and after."""
    import numpy as np
    w = st.w
    st.replica_load.zero_()
    st.assign()
    st.load()
    torch.cuda.synchronize()
    rl = st.replica_load.cpu().numpy().view(np.uint32).astype(np.float32)
    before = rl.sum(0)
    t0 = time.perf_counter()
    table, owner, pred = B.cobalt_intra_node_rebalance(w.N, w.g, w.E, st.table.shape[1],
                                                       st.table, st.owner, rl)
    host_ms = (time.perf_counter() - t0) * 1e3
    L = B.cobalt_layout_create(w.N, w.g, w.E, table.shape[1], table, owner)
    a = torch.empty_like(st.assigned)
    B.cobalt_assign(L, st.topk, st.src, st.seed, st.step, 0, a)
    after = torch.bincount(a.flatten().long(), minlength=w.G).float().cpu().numpy()
    B.cobalt_layout_destroy(L)
    mean = w.T * w.K / w.G
    return {"imbalance_before": float(before.max() / mean),
            "imbalance_predicted": float(pred.max() / mean),
            "imbalance_after": float(after.max() / mean), "host_ms": host_ms}


def drift_with_stage2(st, w, routes, first_layout, replan, fns, torch, B, decay=0.9):
    """The drift cycle once more, untimed, with Stage 2 (Section 3.2) after
    every step: the step's per-replica loads w_er fold into a GPU EMA
    (started from the first step's counts, and from the planned division
    w'_er after the Stage-1 re-plan), and the host rebalancing turns the EMA
    into the layout of the next step. Reports Eq. 1's V and the rank-load
    imbalance of each step's assignment, averaged before and after the
    re-plan."""
    import numpy as np
    st.set_layout(*first_layout)
    st.coact.zero_()
    st.count.zero_()
    st.replica_load.zero_()
    rema = torch.zeros(w.E, w.G, dtype=torch.float32, device=st.device)
    per_step, host_ms = [], []
    for s_ in range(w.steps):
        flags = B.EMA_CLEAR
        if s_ == 0:
            flags |= B.EMA_INIT
        if s_ == w.swap_step:
            torch.cuda.synchronize()
            rema.copy_(torch.from_numpy(replan(s_)))
        st.topk, st.gates = routes[s_]
        st.step = s_
        for f in fns[:-2]:  # statistics, EMA and assignment
            f()
        rn32 = st.remote.to(torch.int32) & 0xFFFF
        V = sum(((rn32 >> n) & 1).sum().item() for n in range(w.N))
        per_rank = torch.bincount(st.assigned.flatten().long(), minlength=w.G).float()
        per_step.append((int(V), float(per_rank.max() / per_rank.mean())))
        st.load()
        B.cobalt_count_ema(st.replica_load, decay, flags, rema)
        rl = rema.cpu().numpy()
        t0 = time.perf_counter()
        table, owner, _ = B.cobalt_intra_node_rebalance(w.N, w.g, w.E, st.table.shape[1],
                                                        st.table, st.owner, rl)
        host_ms.append((time.perf_counter() - t0) * 1e3)
        # the EMA follows the replicas: Algorithm 1 splits a node's tasks of
        # an expert evenly over its replicas there, so each new replica gets
        # the node's total for the expert divided by their number
        held_old = np.zeros((w.E, w.G), bool)
        held_new = np.zeros((w.E, w.G), bool)
        for r in range(w.G):
            held_old[[e for e in st.table[r] if e >= 0], r] = True
            held_new[[e for e in table[r] if e >= 0], r] = True
        node_sum = np.where(held_old, rl, 0.0).reshape(w.E, w.N, w.g).sum(2)
        k_new = held_new.reshape(w.E, w.N, w.g).sum(2)
        share = np.divide(node_sum, k_new, out=np.zeros_like(node_sum), where=k_new > 0)
        remap = np.where(held_new, np.repeat(share, w.g, axis=1), 0.0).astype(np.float32)
        rema.copy_(torch.from_numpy(remap))
        st.set_layout(table, owner)
    before, after = per_step[:w.swap_step], per_step[w.swap_step:]
    return {"ema_decay": decay,
            "mean_V_before": sum(v for v, _ in before) / len(before),
            "mean_V_after": sum(v for v, _ in after) / len(after),
            "mean_imbalance_before": sum(i for _, i in before) / len(before),
            "mean_imbalance_after": sum(i for _, i in after) / len(after),
            "rebalance_host_ms": sum(host_ms) / len(host_ms)}


def stage1_demo(st, torch, B):
    """Periodic global planning (Section 3.2, Stage 1) from the EMAs the GPU
    keeps: the host planner turns ema_coact / ema_count into a layout, and
    this step is re-assigned on it with Algorithm 1. Reports Eq. 1's V and
    the rank-load imbalance (max / mean) against the current layout, then
    after one Stage-2 rebalance of the planned layout on its measured
    replica loads."""
    import numpy as np
    w = st.w

    def measure(table, owner):
        L = B.cobalt_layout_create(w.N, w.g, w.E, table.shape[1], table, owner)
        a = torch.empty_like(st.assigned)
        rn = torch.empty_like(st.remote)
        B.cobalt_assign(L, st.topk, st.src, st.seed, st.step, 0, a, rn)
        load = torch.zeros(w.E, w.G, dtype=torch.int32, device="cuda")
        B.cobalt_replica_load(st.topk, a, w.E, w.G, load, st.load_workspace)
        torch.cuda.synchronize()
        B.cobalt_layout_destroy(L)
        rn32 = rn.to(torch.int32) & 0xFFFF
        V = sum(((rn32 >> n) & 1).sum().item() for n in range(w.N))
        per_rank = torch.bincount(a.flatten().long(), minlength=w.G).float()
        return int(V), float(per_rank.max() / per_rank.mean()), load.cpu().numpy().view(np.uint32)

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    table, owner, plan, obj, feasible = B.cobalt_plan_layout(
        w.N, w.g, w.E, w.S, st.ema_coact, st.ema_count, 0.15)
    host_ms = (time.perf_counter() - t0) * 1e3
    V0, imb0, _ = measure(st.table, st.owner)
    V1, imb1, rl = measure(table, owner)
    t2, o2, _ = B.cobalt_intra_node_rebalance(w.N, w.g, w.E, table.shape[1], table, owner,
                                              rl.astype(np.float32))
    V2, imb2, _ = measure(t2, o2)
    return {"eps": 0.15, "objective": obj, "plan_within_cap": feasible,
            "planner_host_ms": host_ms,
            "current_layout": {"V": V0, "imbalance": imb0},
            "planned_layout": {"V": V1, "imbalance": imb1},
            "planned_then_stage2": {"V": V2, "imbalance": imb2}}


def cpu_baseline(st, n_tokens, torch, W, PL):
    """The oracle, as it stands, on the first n_tokens of the same workload,
    in chunks of 4096 tokens (each chunk a full pass: stats, assign, dispatch
    with packed rows, combine). Single-threaded C."""
    import numpy as np

    import oracle

    w = st.w
    tabs = oracle.layout_tables(w.N, w.g, w.E, st.table, st.owner)
    src_all = W.contiguous_src(w.T, w.G)
    chunk = 4096
    n_tokens = min(n_tokens, w.T)
    steps = {"stats": 0.0, "assign": 0.0, "dispatch": 0.0, "combine": 0.0}
    done = 0
    # the oracle is single-threaded; the thread runs pinned to one host core
    old_aff = os.sched_getaffinity(0)
    core = min(old_aff)
    os.sched_setaffinity(0, {core})
    try:
        for t0 in range(0, n_tokens, chunk):
            n = min(chunk, n_tokens - t0)
            topk = st.topk[t0:t0 + n].cpu().numpy()
            gates = st.gates[t0:t0 + n].cpu().numpy()
            src = np.ascontiguousarray(src_all[t0:t0 + n])
            x = PL.bf16_bits(st.x[t0:t0 + n])
            eo = PL.bf16_bits(st.eo[t0 * w.K:(t0 + n) * w.K])
            c0 = time.perf_counter()
            oracle.coact_stats(topk, w.E)
            c1 = time.perf_counter()
            a, _ = oracle.assign(w.N, w.g, w.E, tabs, topk, src, seed=st.seed, step=0)
            c2 = time.perf_counter()
            _, _, pos, _ = oracle.dispatch(a, w.G, src, x)
            c3 = time.perf_counter()
            oracle.combine(eo, pos, gates)
            c4 = time.perf_counter()
            for k, dt in zip(steps, (c1 - c0, c2 - c1, c3 - c2, c4 - c3)):
                steps[k] += dt
            done += n
    finally:
        os.sched_setaffinity(0, old_aff)
    total = sum(steps.values())
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    return {"value": done / total, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"first {done} tokens of the same workload in chunks of {chunk} "
                      f"(stats, assign, dispatch with packed rows, combine), "
                      f"{total:.1f} s on one host core (core {core}, pinned)",
            "seconds_per_step": {k: round(v, 3) for k, v in steps.items()},
            "host_cpu": model, "host_cpus": os.cpu_count()}


def run_workload(w, seed, steps, warmup, args, full, torch, B, PL, W):
    """Times `steps` steps of workload w after `warmup` untimed ones and
    returns the report. full=False keeps the timing, the roofline figures and
    the routing quality; full=True adds the graph replay, the calls outside
    the step, the HBM references, the node-deduplicated forms, the planner
    demonstrations and the oracle's CPU baseline."""
    wl_name = f"t{w.T}_e{w.E}_k{w.K}_d{w.d}"
    st = PL.RoutingStep(w, seed=seed, device="cuda", expert_out="independent")
    stream = torch.cuda.Stream()
    calls = ["cobalt_coact_stats", "cobalt_assign", "cobalt_dispatch_pack", "cobalt_combine"]
    fns = [st.stats, st.assign, st.pack, st.combine]
    drift = w.steps > 1
    planner = drift and args.replan == "planner"
    if planner:
        # the step also folds its counts into the planner EMAs (and clears
        # them), which the Stage-1 planner reads before the swap step
        def ema_step(stream=None):
            st.ema(0.9, B.EMA_CLEAR | (B.EMA_INIT if st.step == 0 else 0), stream=stream)
        calls.insert(1, "cobalt_coact_ema")
        fns.insert(1, ema_step)

    # a streaming kernel of known size (reads 1 GiB, writes 1 GiB), the
    # reference against which HBM counter readings are scaled
    calib = torch.zeros(1 << 28, dtype=torch.int32, device="cuda")
    calib_dst = torch.empty_like(calib)
    with torch.cuda.stream(stream):
        torch.bitwise_not(calib, out=calib_dst)
    torch.cuda.synchronize()
    del calib, calib_dst

    with torch.cuda.stream(stream):
        for _ in range(warmup):
            for f in fns:
                f(stream=stream)
    torch.cuda.synchronize()
    assert int(st.offsets[-1].item()) == w.T * w.K, "dispatch placed the wrong number of rows"

    # A multi-step (drift) workload cycles through its per-step routings:
    # statistics accumulate over a cycle and the replicas are re-planned
    # from them before the swap step. The re-plan is host work between
    # steps, so such runs are timed by the sum of per-step HIP events.
    plan_info = []

    def replan(s):
        """The layout swap before step s: the Stage-1 planner on the EMAs, or
        the workload's hot-order recipe on the accumulated expert counts."""
        if planner:
            tp = time.perf_counter()
            table, owner, plan, obj, within = B.cobalt_plan_layout(
                w.N, w.g, w.E, w.S, st.ema_coact, st.ema_count, 0.15)
            plan_info.append(((time.perf_counter() - tp) * 1e3, obj, within))
            st.set_layout(table, owner)
            return plan
        else:
            counts = st.count.cpu().numpy().view("uint32").astype("int64")
            hot = sorted(range(w.E), key=lambda e: (-counts[e], e))
            st.set_layout(*W.layout(w, seed, hot_order=hot, plan=s))

    if drift:
        routes = [W.routing(w, seed, step=s, device="cuda") for s in range(w.steps)]
        first_layout = (st.table, st.owner)
        st.coact.zero_()
        st.count.zero_()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(fns) + 1)]
           for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    with torch.cuda.stream(stream):
        for k in range(steps):
            if drift:
                s = k % w.steps
                if s == 0 and k > 0:
                    st.coact.zero_()
                    st.count.zero_()
                    stream.synchronize()
                    st.set_layout(*first_layout)
                if s == w.swap_step:
                    stream.synchronize()
                    replan(s)
                st.topk, st.gates = routes[s]
                st.step = s
            e = evs[k]
            e[0].record(stream)
            for i, f in enumerate(fns):
                f(stream=stream)
                e[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if drift:
        wall = sum(e[0].elapsed_time(e[-1]) for e in evs) * 1e-3

    step_ms = sorted(e[0].elapsed_time(e[-1]) for e in evs)

    def pct(q):
        return step_ms[min(len(step_ms) - 1, int(round(q * (len(step_ms) - 1))))]

    call_ms = {c: 0.0 for c in calls}
    for e in evs:
        for i, c in enumerate(calls):
            call_ms[c] += e[i].elapsed_time(e[i + 1]) / steps
    ab = algorithmic_bytes(w)
    dominant = max(("cobalt_dispatch_pack", "cobalt_combine"), key=lambda c: call_ms[c])
    achieved = ab[dominant] / (call_ms[dominant] * 1e-3)
    traffic = measured_traffic(dominant, wl_name)
    pc_bytes = ab["cobalt_dispatch_pack"] + ab["cobalt_combine"]
    pc_s = (call_ms["cobalt_dispatch_pack"] + call_ms["cobalt_combine"]) * 1e-3
    step_bytes = sum(ab[c] for c in calls)

    result = {
        "metric": METRIC,
        "value": w.T * steps / wall,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": wall * 1e3 / steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"co-activation routing step, {w.describe()}, "
                               f"{w.name}, seed {seed}" +
                               (f", {w.steps}-step drift cycle with re-plan before step "
                                f"{w.swap_step} by the " +
                                ("Stage-1 planner from the EMA statistics (EMA update in "
                                 "each step)" if planner else "hot-order recipe") +
                                ", timed by per-step events" if drift else ""),
                   "T": w.T, "E": w.E, "K": w.K, "d": w.d, "nodes": w.N,
                   "gpus_per_node": w.g, "slots_per_gpu": w.S,
                   "parallelism": "single GPU; virtual ranks are HBM buffers"},
        "roofline": {"bound": "hbm", "kernel": dominant, "achieved": achieved / 1e9,
                     "peak": HBM_PEAK / 1e9, "unit": "GB/s", "frac": achieved / HBM_PEAK,
                     "traffic": traffic},
        "pack_combine_hbm_frac": pc_bytes / pc_s / HBM_PEAK,
        "step_hbm_frac": step_bytes / (wall / steps) / HBM_PEAK,
        "step_ms_percentiles": {"p10": pct(0.1), "median": pct(0.5), "p90": pct(0.9),
                                "note": "per-step HIP events; value uses the wall clock"},
        "device": device_info(torch),
        "call_ms": call_ms,
        "call_gbps": {c: ab[c] / (call_ms[c] * 1e-3) / 1e9 for c in calls},
    }
    if drift:
        # one more cycle, untimed, recording Eq. 1's V and the rank-load
        # imbalance of every step on the layout the cycle's re-plan chose
        st.set_layout(*first_layout)
        st.coact.zero_()
        st.count.zero_()
        per_step = []
        tally = RoutingTally(w, seed, torch, B, W)
        for s_ in range(w.steps):
            if s_ == w.swap_step:
                torch.cuda.synchronize()
                replan(s_)
            st.topk, st.gates = routes[s_]
            st.step = s_
            for f in fns[:-2]:  # statistics, EMA and assignment
                f()
            tally.add(st.layout, st.topk, s_)
            rn32 = st.remote.to(torch.int32) & 0xFFFF
            V = sum(((rn32 >> n) & 1).sum().item() for n in range(w.N))
            per_rank = torch.bincount(st.assigned.flatten().long(), minlength=w.G).float()
            per_step.append((int(V), float(per_rank.max() / per_rank.mean())))
        cycle_ms = [0.0] * w.steps
        for k, e in enumerate(evs):
            cycle_ms[k % w.steps] += e[0].elapsed_time(e[-1]) / sum(
                1 for kk in range(steps) if kk % w.steps == k % w.steps)
        result["cycle_step_ms"] = [round(v, 4) for v in cycle_ms]
        before, after = per_step[:w.swap_step], per_step[w.swap_step:]
        result["replan"] = {"method": "stage1_planner" if planner else "hot_order_recipe",
                            "before_step": w.swap_step,
                            "mean_V_before": sum(v for v, _ in before) / len(before),
                            "mean_V_after": sum(v for v, _ in after) / len(after),
                            "mean_imbalance_before": sum(i for _, i in before) / len(before),
                            "mean_imbalance_after": sum(i for _, i in after) / len(after)}
        if plan_info:
            result["replan"].update({
                "planner_host_ms": sum(p[0] for p in plan_info) / len(plan_info),
                "objective": plan_info[-1][1], "plan_within_cap": plan_info[-1][2]})
        result["routing"] = tally.report()
        result["routing"]["note"] = ("summed over the cycle's steps, each on the layout it ran "
                                     "on (re-planned before step %d)" % w.swap_step)
        tally.close()
    else:
        result["routing"] = routing_quality(st, torch, B, W)
    if not full:
        st.close()
        return result

    if not drift and not args.no_graph:
        # the same four calls captured once as a HIP graph and replayed
        g = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            st.run()
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        tg = time.perf_counter()
        for _ in range(steps):
            g.replay()
        torch.cuda.synchronize()
        wg = time.perf_counter() - tg
        result["graph_replay"] = {"value": w.T * steps / wg, "unit": "tokens/s",
                                  "ms_per_step": wg * 1e3 / steps}
        del g
    # calls outside the step: per-replica load counts (the Stage-2 input)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    with torch.cuda.stream(stream):
        st.load(stream=stream)
        ev[0].record(stream)
        for _ in range(steps):
            st.load(stream=stream)
        ev[1].record(stream)
    torch.cuda.synchronize()
    result["extra_calls_ms"] = {"cobalt_replica_load": ev[0].elapsed_time(ev[1]) / steps}
    ref = hbm_reference(torch, stream, st)
    result["hbm_reference"] = ref
    # the combine's floor: its row loads at the gather rate, then y at the fill rate
    y_ms = w.T * w.d * 2 / (ref["write_fill"]["GB_s"] * 1e9) * 1e3
    result["call_vs_ceiling"] = {
        "cobalt_dispatch_pack_vs_write_fill":
            result["call_gbps"]["cobalt_dispatch_pack"] / ref["write_fill"]["GB_s"],
        "pack_store_ceiling_ms": ref["pack_store"]["ms"],
        "cobalt_dispatch_pack_ms": call_ms["cobalt_dispatch_pack"],
        "cobalt_dispatch_pack_time_vs_store_ceiling":
            ref["pack_store"]["ms"] / call_ms["cobalt_dispatch_pack"],
        "combine_floor_ms": ref["gather_read"]["ms"] + y_ms,
        "cobalt_combine_ms": call_ms["cobalt_combine"],
        "cobalt_combine_time_vs_floor": (ref["gather_read"]["ms"] + y_ms) / call_ms["cobalt_combine"],
        "note": "time ratios: the ceiling's time over the call's (1.0 = at the ceiling)"}
    # the node-deduplicated dispatch of the last step's assignment: one row
    # per (token, destination node) instead of one per (token, expert)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    with torch.cuda.stream(stream):
        st.node_pack(stream=stream)
        ev[0].record(stream)
        for _ in range(steps):
            st.node_pack(stream=stream)
        ev[1].record(stream)
    torch.cuda.synchronize()
    node_ms = ev[0].elapsed_time(ev[1]) / steps
    rows = int(st.node_offsets[-1].item())
    home = (torch.arange(w.T, device="cuda") // (w.T // w.G)) // w.g if st.src is None \
        else st.src.long() // w.g
    local_rows = int((st.node_pos.gather(1, home.long()[:, None]) >= 0).sum().item())
    nb = node_dispatch_bytes(w, rows)
    result["extra_calls_ms"]["cobalt_node_dispatch_pack"] = node_ms
    result["node_dedup_dispatch"] = {
        "rows": rows, "rows_per_token": rows / w.T, "cross_node_rows": rows - local_rows,
        "rows_vs_pair_layout": rows / (w.T * w.K),
        "algorithmic_bytes": nb, "achieved_gbps": nb / (node_ms * 1e-3) / 1e9,
        "hbm_frac": nb / (node_ms * 1e-3) / HBM_PEAK,
        "traffic": measured_traffic("cobalt_node_dispatch_pack", wl_name),
        "pair_pack_ms": call_ms["cobalt_dispatch_pack"], "node_pack_ms": node_ms}
    # its reverse: per-(token, node) partial sums, then the source-side sum
    with torch.cuda.stream(stream):
        st.node_combine(stream=stream)
        ev[0].record(stream)
        for _ in range(steps):
            st.node_combine(stream=stream)
        ev[1].record(stream)
    torch.cuda.synchronize()
    ncb_ms = ev[0].elapsed_time(ev[1]) / steps
    cb = node_combine_bytes(w, rows)
    result["extra_calls_ms"]["cobalt_node_combine"] = ncb_ms
    result["node_dedup_combine"] = {
        "algorithmic_bytes": cb, "achieved_gbps": cb / (ncb_ms * 1e-3) / 1e9,
        "hbm_frac": cb / (ncb_ms * 1e-3) / HBM_PEAK, "node_combine_ms": ncb_ms,
        "pair_combine_ms": call_ms["cobalt_combine"],
        "cross_node_rows": rows - local_rows}
    # the step as a node-deduplicating transport would run it: statistics,
    # assignment, node-deduplicated pack and node-level combine
    def node_step():
        st.stats(stream=stream)
        st.assign(stream=stream)
        st.node_pack(stream=stream)
        st.node_combine(stream=stream)
    with torch.cuda.stream(stream):
        node_step()
        ev[0].record(stream)
        for _ in range(steps):
            node_step()
        ev[1].record(stream)
    torch.cuda.synchronize()
    nstep_ms = ev[0].elapsed_time(ev[1]) / steps
    result["node_dedup_step"] = {"ms_per_step": nstep_ms, "value": w.T / (nstep_ms * 1e-3),
                                 "unit": "tokens/s",
                                 "calls": "stats + assign + node_dispatch_pack + node_combine"}
    # planner statistics of one step: EMA update of the co-activation and
    # expert counts, and the Ochiai similarity (the Fig. 3 statistic)
    st.coact.zero_()
    st.count.zero_()
    with torch.cuda.stream(stream):
        st.stats(stream=stream)
        st.ema(0.9, B.EMA_INIT, stream=stream)
        ev[0].record(stream)
        for _ in range(steps):
            st.ema(0.9, 0, stream=stream)
        ev[1].record(stream)
    torch.cuda.synchronize()
    result["extra_calls_ms"]["cobalt_coact_ema"] = ev[0].elapsed_time(ev[1]) / steps
    pairs = torch.triu(st.coact != 0, diagonal=1)
    result["planner_statistics"] = {
        "ochiai_mean_coactivated_pairs": float(st.ochiai[pairs].mean().item()),
        "coactivated_pairs": int(pairs.sum().item()),
        "pairs": w.E * (w.E - 1) // 2}
    cl = W.clusters(w, seed)
    if cl is not None:
        same = torch.zeros(w.E, w.E, dtype=torch.bool, device="cuda")
        idx = torch.from_numpy(cl).cuda()
        same[idx[:, :, None], idx[:, None, :]] = True
        inside = pairs & same
        result["planner_statistics"]["ochiai_mean_planted_cluster_pairs"] = \
            float(st.ochiai[inside].mean().item())
        result["planner_statistics"]["ochiai_mean_other_pairs"] = \
            float(st.ochiai[pairs & same.logical_not()].mean().item())
    result["routing"]["stage2_rebalance"] = stage2_demo(st, torch, B, W)
    result["routing"]["stage1_plan"] = stage1_demo(st, torch, B)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(st, args.cpu_sample_tokens, torch, W, PL)
    if planner:
        # last, since it leaves another layout and assignment behind
        result["replan"]["with_stage2_each_step"] = drift_with_stage2(
            st, w, routes, first_layout, replan, fns, torch, B)
    st.close()
    return result


ROUTING_KEYS = ("alg1", "owner_only", "contiguous_ep_owner_only", "V_reduction_vs_owner_only",
                "V_reduction_vs_contiguous_ep_owner_only", "steps_summed", "alg1_V_per_step",
                "note")


def summarize(r):
    """The per-workload entry of the report."""
    out = {"config": r["config"]["workload"], "tokens_per_s": r["value"],
           "ms_per_step": r["ms_per_step"], "steps": r["steps"], "warmup": r["warmup"],
           "step_ms_median": r["step_ms_percentiles"]["median"],
           "pack_combine_hbm_frac": r["pack_combine_hbm_frac"],
           "step_hbm_frac": r["step_hbm_frac"], "call_ms": r["call_ms"],
           "routing": {k: v for k, v in r["routing"].items() if k in ROUTING_KEYS}}
    for k in ("cycle_step_ms", "replan"):
        if k in r:
            out[k] = r[k]
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the library has "
              "no inter-GPU collectives; its virtual ranks are buffers on one GPU", file=sys.stderr)
        sys.exit(2)
    import gc

    import torch

    from paper_2609_36959_amd import binding as B
    from paper_2609_36959_amd import pipeline as PL
    from paper_2609_36959_amd import workload as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    B.lib()
    w = W.WORKLOADS[args.workload]
    seed = w.seed if args.seed is None else args.seed
    print(f"bench: {w.name} ({w.describe()}), {args.steps} steps", file=sys.stderr, flush=True)
    result = run_workload(w, seed, args.steps, args.warmup, args, True, torch, B, PL, W)
    if not args.headline_only:
        # every seeded workload once more, each at its default seed: the
        # single-step ones over the same number of steps, the drift workload
        # over one full cycle
        wl = {}
        names = W.NAMES if args.workloads == "all" else args.workloads.split(",")
        for name in names:
            if name == args.workload and args.seed is None:
                wl[name] = summarize(result)
                continue
            gc.collect()
            torch.cuda.empty_cache()
            ow = W.WORKLOADS[name]
            n = ow.steps if ow.steps > 1 else args.steps
            print(f"bench: {name} ({ow.describe()}), {n} steps", file=sys.stderr, flush=True)
            wl[name] = summarize(run_workload(ow, ow.seed, n, args.warmup, args, False, torch, B,
                                              PL, W))
        result["workloads"] = wl
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
