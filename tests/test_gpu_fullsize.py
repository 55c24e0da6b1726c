"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times (RoutingStep, independent expert outputs). Integer outputs
(statistics, assignment, counts, offsets, pos) are compared in full against
the oracle; packed rows and combined rows are compared on seeded samples the
oracle computes one by one; the dispatch/combine round trip (expert outputs
= packed rows, gates summing to one, so y = x) is checked on every row."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36959_amd import binding as B
from paper_2609_36959_amd import pipeline as PL
from paper_2609_36959_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    B.lib()
    yield
    torch.cuda.empty_cache()


def check_step(st, tabs, C_ref, cnt_ref, rng, n_rows=4096, n_tok=256):
    """Compares one step's outputs with the oracle; returns the oracle's
    accumulated statistics."""
    w = st.w
    topk = st.topk.cpu().numpy()
    gates = st.gates.cpu().numpy()
    a, rn = oracle.assign(w.N, w.g, w.E, tabs, topk, None, seed=st.seed, step=st.step)
    assert np.array_equal(st.assigned.cpu().numpy(), a), "assignment differs"
    assert np.array_equal(st.remote.cpu().numpy().view(np.uint16), rn), "remote nodes differ"
    counts, offsets, pos, _ = oracle.dispatch(a, w.G)
    assert np.array_equal(st.counts.cpu().numpy(), counts)
    assert np.array_equal(st.offsets.cpu().numpy(), offsets)
    assert np.array_equal(st.pos.cpu().numpy(), pos), "pos differs"
    C_ref, cnt_ref = oracle.coact_stats(topk, w.E, C_ref, cnt_ref)
    assert np.array_equal(st.coact.cpu().numpy().view(np.uint32), C_ref)
    assert np.array_equal(st.count.cpu().numpy().view(np.uint32), cnt_ref)

    # packed rows: packed[pos[p]] must be x[t] bit for bit
    p = rng.choice(w.T * w.K, size=min(n_rows, w.T * w.K), replace=False)
    rows = torch.from_numpy(pos.ravel()[p].astype(np.int64)).cuda()
    toks = torch.from_numpy(p // w.K).cuda()
    assert np.array_equal(PL.bf16_bits(st.packed[rows]), PL.bf16_bits(st.x[toks]))

    # combined rows: the oracle's weighted sum of the expert rows the
    # oracle's pos selects
    t = np.sort(rng.choice(w.T, size=min(n_tok, w.T), replace=False))
    sel = pos[t].ravel().astype(np.int64)
    eo_rows = PL.bf16_bits(st.eo[torch.from_numpy(sel).cuda()])
    ident = np.arange(len(t) * w.K, dtype=np.int32).reshape(len(t), w.K)
    y_ref, _ = oracle.combine(eo_rows, ident, gates[t])
    assert np.array_equal(PL.bf16_bits(st.y[torch.from_numpy(t).cuda()]), y_ref)
    return C_ref, cnt_ref


def round_trip(st):
    """Combine of the packed rows themselves returns x on every row."""
    y = torch.empty_like(st.y)
    B.cobalt_combine(st.packed, st.pos, st.gates, y)
    torch.cuda.synchronize()
    assert torch.equal(y.float(), st.x.float())


@pytest.mark.parametrize("name", ["clusters-e64", "colocate-e128", "colocate-e256"])
def test_full_size_single_step(name):
    w = W.WORKLOADS[name]
    print(f"full size {name} {w.describe()}", flush=True)
    st = PL.RoutingStep(w, seed=w.seed, device="cuda")
    st.run()
    st.load()
    torch.cuda.synchronize()
    tabs = oracle.layout_tables(w.N, w.g, w.E, st.table, st.owner)
    check_step(st, tabs, None, None, np.random.default_rng(w.seed))
    ref = oracle.replica_load(st.topk.cpu().numpy(), st.assigned.cpu().numpy(), w.E, w.G)
    assert np.array_equal(st.replica_load.cpu().numpy().view(np.uint32), ref)
    round_trip(st)
    st.close()
    del st
    torch.cuda.empty_cache()


def test_drift_sixteen_steps_with_layout_swap():
    """16 steps of T=262144, E=384: statistics accumulate across steps, the
    Zipf skew drifts every step, and before step 8 the replicas are
    re-planned from the accumulated expert counts."""
    w = W.WORKLOADS["drift-e384"]
    seed = w.seed
    st = PL.RoutingStep(w, seed=seed, device="cuda")
    rng = np.random.default_rng(44)
    tabs = oracle.layout_tables(w.N, w.g, w.E, st.table, st.owner)
    C_ref = cnt_ref = None
    for step in range(w.steps):
        if step == w.swap_step:
            gpu_hot = np.argsort(-st.count.cpu().numpy().view(np.uint32).astype(np.int64),
                                 kind="stable")
            ref_hot = np.argsort(-cnt_ref.astype(np.int64), kind="stable")
            assert np.array_equal(gpu_hot, ref_hot)
            table, owner = W.layout(w, seed, hot_order=gpu_hot, plan=step)
            st.set_layout(table, owner)
            tabs = oracle.layout_tables(w.N, w.g, w.E, *W.layout(w, seed, hot_order=ref_hot,
                                                                  plan=step))
        if step > 0:
            st.set_routing(step)
        st.run()
        torch.cuda.synchronize()
        print(f"drift step {step}", flush=True)
        C_ref, cnt_ref = check_step(st, tabs, C_ref, cnt_ref, rng, n_rows=1024, n_tok=64)
    round_trip(st)
    assert cnt_ref.sum() == w.steps * w.T * w.K
    st.close()
    del st
    torch.cuda.empty_cache()


def test_drift_cycle_with_the_stage1_planner():
    """The method's own loop over the drift workload's 16 steps (T=262144,
    E=384): each step's counts fold into the EMAs on the GPU and are
    cleared; before step 8 the host planner turns the EMAs into a new
    layout; Algorithm 1 and the dispatch layout run on it. The oracle runs
    the same loop from its own counts; every integer output, the EMAs and
    the planned layout agree exactly."""
    w = W.WORKLOADS["drift-e384"]
    seed = w.seed
    st = PL.RoutingStep(w, seed=seed, device="cuda")
    ref_c = np.zeros((w.E, w.E), np.float32)
    ref_n = np.zeros(w.E, np.float32)
    tabs = oracle.layout_tables(w.N, w.g, w.E, st.table, st.owner)
    for step in range(w.steps):
        if step > 0:
            st.set_routing(step)
        topk = st.topk.cpu().numpy()
        if step == w.swap_step:
            got = B.cobalt_plan_layout(w.N, w.g, w.E, w.S, st.ema_coact, st.ema_count, 0.15)
            want = oracle.plan_layout(w.N, w.g, w.E, w.S, ref_c, ref_n, 0.15)
            for x, y in zip(got[:3], want[:3]):
                assert np.array_equal(x, y), "planned layout differs"
            assert got[3] == want[3] and got[4] == want[4]
            st.set_layout(got[0], got[1])
            tabs = oracle.layout_tables(w.N, w.g, w.E, want[0], want[1])
        st.stats()
        st.ema(0.9, B.EMA_CLEAR | (B.EMA_INIT if step == 0 else 0))
        st.assign()
        st.pack()
        torch.cuda.synchronize()
        print(f"planner cycle step {step}", flush=True)
        C, n = oracle.coact_stats(topk, w.E)
        oracle.count_ema(C, 0.9, ema=ref_c, init=step == 0)
        oracle.count_ema(n, 0.9, ema=ref_n, init=step == 0)
        assert np.array_equal(st.ema_coact.cpu().numpy().view(np.uint32), ref_c.view(np.uint32))
        assert np.array_equal(st.ema_count.cpu().numpy().view(np.uint32), ref_n.view(np.uint32))
        a, rn = oracle.assign(w.N, w.g, w.E, tabs, topk, None, seed=seed, step=step)
        assert np.array_equal(st.assigned.cpu().numpy(), a), f"assignment differs at {step}"
        assert np.array_equal(st.remote.cpu().numpy().view(np.uint16), rn)
        counts, offsets, pos, _ = oracle.dispatch(a, w.G)
        assert np.array_equal(st.offsets.cpu().numpy(), offsets)
        assert np.array_equal(st.pos.cpu().numpy(), pos)
    st.close()
    del st
    torch.cuda.empty_cache()
