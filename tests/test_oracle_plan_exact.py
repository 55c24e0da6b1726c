"""Pins of the oracle's exact Stage-1 solver (Section 3.2, Eq. 3, and the
MILP of the appendix) on tiny instances: optima worked by hand, the returned
layout checked against Eq. 3's constraints with its work division found by
a linear program (not by the solver's own feasibility rule), and the
optimum compared with the appendix's MILP solved by scipy's HiGHS."""
import itertools

import numpy as np
import pytest
from scipy.optimize import linprog

import oracle
from test_oracle_plan_milp import eq3_milp


def sym(E, pairs):
    c = np.zeros((E, E), np.float32)
    for i, j, v in pairs:
        c[i, j] = c[j, i] = v
    return c


def division_lp(table, w, cap, E):
    """Is there a work division within cap on this layout? Solved as a
    transport LP over the variables l_er of the held (e, r)."""
    G = table.shape[0]
    var = [(e, r) for r in range(G) for e in table[r] if e >= 0]
    if not var:
        return False
    A_eq = np.zeros((E, len(var)))
    A_ub = np.zeros((G, len(var)))
    for k, (e, r) in enumerate(var):
        A_eq[e, k] = 1.0
        A_ub[r, k] = 1.0
    res = linprog(np.zeros(len(var)), A_ub=A_ub, b_ub=np.full(G, cap * (1 + 1e-9)),
                  A_eq=A_eq, b_eq=w.astype(np.float64), bounds=(0, None), method="highs")
    return res.status == 0


def check_layout(N, g, E, S, c, w, eps, obj, table):
    """Eq. 3's constraints and objective from the returned layout alone."""
    G = N * g
    assert table.shape == (G, S)
    held = np.zeros((E, G), bool)
    for r in range(G):
        ids = [int(e) for e in table[r] if e >= 0]
        assert len(ids) == len(set(ids)) and len(ids) <= S
        held[ids, r] = True
    assert held.any(1).all()
    on = held.reshape(E, N, g).any(2)
    want = sum(float(c[i, j]) for n in range(N) for i in range(E) for j in range(i + 1, E)
               if on[i, n] and on[j, n])
    assert obj == pytest.approx(want, rel=1e-12, abs=1e-12)
    cap = (1.0 + float(np.float32(eps))) * float(w.astype(np.float64).sum()) / G
    assert division_lp(table, w, cap, E)


def test_two_pairs_on_two_nodes():
    """One rank per node, two slots each: the optimum puts each co-activated
    pair on its own node, 10 + 10."""
    c = sym(4, [(0, 1, 10), (2, 3, 10)])
    w = np.ones(4, np.float32)
    found, obj, table = oracle.plan_exact(2, 1, 4, 2, c, w, 0.15)
    assert found and obj == 20.0
    check_layout(2, 1, 4, 2, c, w, 0.15, obj, table)
    # of the two optimal layouts the first in enumeration order (rank 0's
    # set the smaller bitmask) is returned
    assert table.tolist() == [[0, 1], [2, 3]]


def test_a_spare_slot_holds_the_strong_pair_on_both_nodes():
    """A third slot per rank: each node takes one pair plus a replica that
    completes the strong cross pair (0, 2): each node counts 10 + 50, and no
    three experts are worth more (the best triples are {0,1,2} and {0,2,3},
    60 each)."""
    c = sym(4, [(0, 1, 10), (2, 3, 10), (0, 2, 50)])
    w = np.ones(4, np.float32)
    found, obj, table = oracle.plan_exact(2, 1, 4, 3, c, w, 0.15)
    assert found and obj == 120.0
    check_layout(2, 1, 4, 3, c, w, 0.15, obj, table)


def test_the_work_cap_separates_the_heavy_pair():
    """Two heavy experts (work 10) that co-activate most, two light ones,
    two ranks of two slots, eps = 0: cap = 22 / 2 = 11, so the heavy pair
    cannot share a rank. Of the layouts that split it, {0,2}|{1,3} is worth
    3 + 4 = 7 and {0,3}|{1,2} 1 + 2 = 3. With eps = 1 the cap is 22 and the
    heavy pair fits together: 10."""
    c = sym(4, [(0, 1, 10), (0, 2, 3), (1, 3, 4), (0, 3, 1), (1, 2, 2)])
    w = np.array([10, 10, 1, 1], np.float32)
    found, obj, table = oracle.plan_exact(2, 1, 4, 2, c, w, 0.0)
    assert found and obj == 7.0
    check_layout(2, 1, 4, 2, c, w, 0.0, obj, table)
    found, obj, _ = oracle.plan_exact(2, 1, 4, 2, c, w, 1.0)
    assert found and obj == 10.0


def test_work_split_over_replicas():
    """One expert carries more than one rank's cap (work 5 of 8, cap 2.3 on
    four ranks at eps 0.15): it needs replicas on three ranks, which the
    slot budget allows only if the light experts share."""
    E = 4
    w = np.array([5, 1, 1, 1], np.float32)
    c = sym(E, [(1, 2, 1), (2, 3, 1)])
    found, obj, table = oracle.plan_exact(2, 2, E, 2, c, w, 0.15)
    assert found
    check_layout(2, 2, E, 2, c, w, 0.15, obj, table)
    held0 = sum(1 for r in range(4) if 0 in table[r])
    assert held0 >= 3
    # one slot per rank leaves no room for a replica: no layout meets the cap
    assert oracle.plan_exact(2, 2, E, 1, c, w, 0.15)[0] is False


def test_infeasible_and_degenerate_cases():
    c = sym(3, [(0, 1, 1)])
    w = np.ones(3, np.float32)
    # two slots in total for three experts: no layout covers them all
    assert oracle.plan_exact(1, 2, 3, 1, c, w, 0.15) == (False, None, None)
    # one node: every pair counts once, whatever the ranks hold
    c4 = sym(4, [(0, 1, 1), (0, 2, 2), (1, 3, 4), (2, 3, 8)])
    found, obj, table = oracle.plan_exact(1, 2, 4, 2, c4, np.ones(4, np.float32), 0.15)
    assert found and obj == 15.0
    # no co-activation: objective 0, any covering layout
    found, obj, _ = oracle.plan_exact(2, 2, 5, 2, np.zeros((5, 5), np.float32),
                                      np.ones(5, np.float32), 0.15)
    assert found and obj == 0.0


def test_only_the_upper_triangle_is_read():
    c = sym(4, [(0, 1, 10), (2, 3, 10)])
    lower = np.tril(c).astype(np.float32)
    lower[2, 3] = 0
    assert oracle.plan_exact(2, 1, 4, 2, np.triu(c), np.ones(4, np.float32), 0.15)[1] == 20.0
    assert oracle.plan_exact(2, 1, 4, 2, lower, np.ones(4, np.float32), 0.15)[1] == 0.0


def test_rejects_sizes_beyond_the_enumeration():
    c = np.zeros((7, 7), np.float32)
    with pytest.raises(oracle.OracleError):
        oracle.plan_exact(2, 2, 7, 3, c, np.ones(7, np.float32), 0.15)
    with pytest.raises(oracle.OracleError):
        oracle.plan_exact(5, 1, 4, 3, c[:4, :4], np.ones(4, np.float32), 0.15)


def tiny_instance(rng, N, E):
    """Pair weights on a 1/4 grid (exact in fp32 and in any sum order),
    clustered by a seeded node label, Pareto work."""
    grp = rng.integers(0, N, size=E)
    c = rng.random((E, E)) * 5
    same = grp[:, None] == grp[None, :]
    c[same] += 40 * rng.random((E, E))[same]
    c = np.triu(c, 1)
    c = np.rint((c + c.T) * 4) / 4
    w = np.rint((rng.pareto(1.5, E) * 50 + 10) * 4) / 4
    return c.astype(np.float32), w.astype(np.float32)


TINY = [(2, 1, 4, 2), (2, 1, 5, 3), (2, 2, 5, 2), (2, 2, 6, 2), (2, 2, 6, 3), (4, 1, 6, 2),
        (3, 1, 6, 3), (1, 4, 6, 2)]


@pytest.mark.parametrize("N,g,E,S", TINY)
def test_optimum_equals_the_appendix_milp(N, g, E, S):
    rng = np.random.default_rng(N * 100 + g * 10 + E + S)
    for trial in range(3):
        c, w = tiny_instance(rng, N, E)
        eps = (0.15, 0.0, 0.5)[trial]
        found, obj, table = oracle.plan_exact(N, g, E, S, c, w, eps)
        ref = eq3_milp(N, g, E, S, c, w, eps, time_limit=30, allow_infeasible=True)
        print(f"N={N} g={g} E={E} S={S} eps={eps}: exact {obj}, MILP {ref}")
        if ref is None:  # no layout meets the cap
            assert not found
            continue
        best, bound = ref
        assert abs(best - bound) <= 1e-6 * max(1.0, abs(bound)), "MILP not solved to optimum"
        assert found
        check_layout(N, g, E, S, c, w, eps, obj, table)
        assert obj == pytest.approx(best, rel=1e-9, abs=1e-9)


def test_brute_force_on_the_smallest_case():
    """N = 2 ranks of one slot pair, E = 3: all 7^2 layouts of subsets of
    size <= 2 listed in Python, feasibility by the LP, best value by hand
    formula."""
    rng = np.random.default_rng(5)
    N, g, E, S = 2, 1, 3, 2
    for _ in range(5):
        c, w = tiny_instance(rng, N, E)
        cap = 1.15 * float(w.astype(np.float64).sum()) / 2
        subsets = [s for k in range(S + 1) for s in itertools.combinations(range(E), k)]
        best = None
        for a, b in itertools.product(subsets, repeat=2):
            if set(a) | set(b) != set(range(E)):
                continue
            table = np.full((2, S), -1, np.int32)
            table[0, :len(a)] = a
            table[1, :len(b)] = b
            if not division_lp(table, w, cap, E):
                continue
            v = sum(float(c[i, j]) for grp in (a, b) for i, j in itertools.combinations(grp, 2))
            best = v if best is None else max(best, v)
        found, obj, _ = oracle.plan_exact(N, g, E, S, c, w, 0.15)
        assert found == (best is not None)
        if found:
            assert obj == best
