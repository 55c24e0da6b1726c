"""The Stage-1 heuristic against the exact problem it approximates: the
appendix's MILP form of Eq. 3, solved with scipy's HiGHS on small seeded
instances. Whenever the heuristic's plan meets the work cap it is a
feasible point of that MILP, so its objective can never exceed the solver's
bound on the optimum; a plan above the bound would mean a wrong objective or
a broken constraint. The heuristic's share of the best MILP solution is
also held above a floor."""
import numpy as np
import pytest
from scipy.optimize import Bounds, LinearConstraint, milp
from scipy.sparse import lil_matrix

import oracle


def eq3_milp(N, g, E, S, c, w, eps, time_limit, allow_infeasible=False):
    """x_er in {0,1}, u_en, z_ijn in [0,1], l_er >= 0 as in the appendix;
    z only for pairs with c_ij > 0 (the others add nothing). Returns (best
    objective, dual bound), or None for an infeasible instance when
    allow_infeasible is set."""
    G = N * g
    pairs = [(i, j) for i in range(E) for j in range(i + 1, E) if c[i, j] > 0]
    nx, nu, nz = E * G, E * N, len(pairs) * N
    ox, ou, oz, ol = 0, nx, nx + nu, nx + nu + nz
    nv = ol + E * G
    rows, lo, hi = [], [], []

    def add(coefs, lo_, hi_):
        rows.append(coefs)
        lo.append(lo_)
        hi.append(hi_)

    for e in range(E):
        for n in range(N):
            for r in range(n * g, (n + 1) * g):
                add({ox + e * G + r: 1, ou + e * N + n: -1}, -np.inf, 0)   # x_er <= u_en
            d = {ou + e * N + n: 1}
            for r in range(n * g, (n + 1) * g):
                d[ox + e * G + r] = -1
            add(d, -np.inf, 0)                                              # u_en <= sum x_er
    for p, (i, j) in enumerate(pairs):
        for n in range(N):
            z = oz + p * N + n
            add({z: 1, ou + i * N + n: -1}, -np.inf, 0)
            add({z: 1, ou + j * N + n: -1}, -np.inf, 0)
            add({z: 1, ou + i * N + n: -1, ou + j * N + n: -1}, -1, np.inf)
    cap = (1.0 + float(np.float32(eps))) * float(w.astype(np.float64).sum()) / G
    for e in range(E):
        add({ox + e * G + r: 1 for r in range(G)}, 1, np.inf)                 # coverage
        add({ol + e * G + r: 1 for r in range(G)}, float(w[e]), float(w[e]))  # work conserved
        for r in range(G):
            add({ol + e * G + r: 1, ox + e * G + r: -float(w[e])}, -np.inf, 0)
    for r in range(G):
        add({ox + e * G + r: 1 for e in range(E)}, -np.inf, S)                # replica budget
        add({ol + e * G + r: 1 for e in range(E)}, -np.inf, cap)              # balance
    A = lil_matrix((len(rows), nv))
    for k, d in enumerate(rows):
        for v, a in d.items():
            A[k, v] = a
    cost = np.zeros(nv)
    for p, (i, j) in enumerate(pairs):
        cost[oz + p * N: oz + p * N + N] = -float(c[i, j])
    integ = np.zeros(nv)
    integ[ox:ox + nx] = 1
    ub = np.ones(nv)
    ub[ol:] = np.inf
    res = milp(cost, constraints=LinearConstraint(A.tocsr(), lo, hi), integrality=integ,
               bounds=Bounds(np.zeros(nv), ub), options={"time_limit": time_limit})
    if res.status == 2 and allow_infeasible:  # HiGHS: the problem is infeasible
        return None
    assert res.x is not None, res.message
    return -res.fun, -res.mip_dual_bound


def instance(rng, N, E):
    grp = rng.integers(0, N, size=E)
    c = rng.random((E, E)) * 5
    same = grp[:, None] == grp[None, :]
    c[same] += 40 * rng.random((E, E))[same]
    c = np.triu(c, 1)
    c = np.rint((c + c.T) * 4) / 4  # multiples of 1/4: the planner's 1/256 grid is exact
    w = (rng.pareto(1.5, E) * 50 + 10).astype(np.float32)
    return c.astype(np.float32), w


@pytest.mark.parametrize("N,g,E,seed", [(2, 2, 8, 0), (2, 2, 10, 1), (2, 2, 12, 2),
                                        (3, 1, 9, 3), (2, 3, 12, 4), (4, 1, 8, 5)])
def test_heuristic_is_within_the_exact_bound(N, g, E, seed):
    rng = np.random.default_rng(seed)
    G = N * g
    S = int(np.ceil(1.5 * E / G))
    c, w = instance(rng, N, E)
    table, owner, plan, obj, feasible = oracle.plan_layout(N, g, E, S, c, w, 0.15)
    best, bound = eq3_milp(N, g, E, S, c, w, 0.15, time_limit=20)
    print(f"N={N} g={g} E={E}: heuristic {obj:.2f}, MILP best {best:.2f}, bound {bound:.2f}, "
          f"share {obj / best:.3f}, within cap {feasible}")
    if feasible:
        assert obj <= bound * (1 + 1e-6) + 1e-6
    assert obj >= 0.7 * best


def test_a_tight_instance_is_brought_within_the_cap():
    """Three nodes of two ranks with two slots each hold nine experts; expert
    0 (work 273) needs more than two ranks at cap = 1.15 * 485 / 6 = 92.958.
    The MILP finds a plan within the cap, so Eq. 3 is feasible here. Step 1
    fills node 0 with expert 0 up to g cap. The repairs inside and across
    nodes then find no rank with room and a free slot. Only the retry with
    work slack on every node reaches the cap."""
    N, g, S, E = 3, 2, 2, 9
    w = np.array([273, 32, 5, 54, 8, 7, 19, 64, 23], np.float32)
    c = np.zeros((E, E), np.float32)
    for i, j, v in [(0, 1, 18), (0, 2, 5), (0, 6, 12), (1, 3, 7), (1, 6, 11), (1, 7, 19),
                    (2, 3, 4), (2, 8, 9), (4, 5, 16), (4, 6, 1)]:
        c[i, j] = c[j, i] = v
    best, bound = eq3_milp(N, g, E, S, c, w, 0.15, time_limit=20)
    table, owner, plan, obj, feasible = oracle.plan_layout(N, g, E, S, c, w, 0.15)
    assert feasible and obj <= bound * (1 + 1e-6) + 1e-6
    cap = 1.15 * float(w.astype(np.float64).sum()) / (N * g)
    loads = plan.astype(np.float64).sum(0)
    assert loads.max() <= cap * (1 + 1e-6)
    held = np.zeros((E, N * g), bool)
    for r in range(N * g):
        ids = [int(e) for e in table[r] if e >= 0]
        assert len(ids) == len(set(ids)) and len(ids) <= S
        held[ids, r] = True
    assert held.any(1).all() and not plan[~held].any()
    assert np.allclose(plan.astype(np.float64).sum(1), w, rtol=1e-5)
