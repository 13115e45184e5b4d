"""Invariants of the method that pin the oracle at sizes brute force cannot reach.

* Floor (Eq. 1): sinks are in no boundary, so every strategy recomputes
  them; with the exact family and B >= 2 M(V) the singleton chain in
  topological order reaches exactly T(Sinks).
* Ceiling (Section 4.4): the memory-centric overhead is at most T(V), and
  equals it once B >= 2 M(V) (the one-segment chain {V} needs 2 M(V)).
* Budget floor: every node lies in some segment V_i, whose Eq. 2 term is at
  least 2 M_v, so B < 2 max M_v has no solution.
* Monotonicity in B (the problem statement): opt_B is pointwise
  non-increasing in B; t* is non-increasing; feasibility is monotone.
* Family inclusion (Section 4.3): the pruned family is a subset of the
  exact one, so its opt rows are pointwise >= on shared sets.
* Row minimum: min_t opt[L, t] equals the least cache memory over all
  feasible chains ending at L, computed here by a separate t-free DP with
  Python bitmask sets.
* Support: opt[L, t] finite implies t <= T(L minus boundary(L)).
"""

import numpy as np
import pytest

from paper_1905_11722_amd import workloads as W
from tests import bruteforce as bf


def INF_as_big(a):
    a = a.astype(np.int64).copy()
    a[a < 0] = np.iinfo(np.int64).max
    return a


def t_free_min_cache(g, mode, B):
    """f[L] = least M(U) over feasible chains ending at L (no t axis)."""
    sg = bf.SetGraph(g)
    F = bf.family(sg, mode)
    f = [None] * len(F)
    f[0] = 0
    bd = [sg.boundary(S) for S in F]
    # Dominance on m alone is exact here: the next segment's memory grows
    # with M(U) and the next cache is U plus new boundary nodes.  Track the
    # set U itself so that M(U) is evaluated from its definition.
    bestU = [None] * len(F)
    bestU[0] = 0
    for j, L2 in enumerate(F):
        for i in range(j):
            L = F[i]
            if bestU[i] is None or L & ~L2 or L == L2:
                continue
            if sg.segment_memory(bestU[i], L, L2) > B:
                continue
            U2 = bestU[i] | bd[j]
            if bestU[j] is None or sg.M(U2) < sg.M(bestU[j]):
                bestU[j] = U2
    return [None if U is None else sg.M(U) for U in bestU], F


GRAPHS = [
    ("rand10", lambda: W.random_dag(10, 0.3, 7)),
    ("rand12", lambda: W.random_dag(12, 0.35, 8)),
    ("layered4x3", lambda: W.layered(4, 3, seed=2, tmax=30, mmax=20)),
    ("ladder6", lambda: W.ladder(6, seed=1, tmax=20, mmax=20)),
    ("chain16", lambda: W.case("chain16").graph),
]


@pytest.mark.parametrize("name,make", GRAPHS)
def test_floor_and_ceiling(oracle_mod, name, make):
    g = make()
    sg = bf.SetGraph(g)
    B = 2 * sum(g.M)
    r = oracle_mod.solve(g, "exact", B, "tc")
    assert r.t_star == sg.T(sg.sinks())
    for mode in ("exact", "pruned"):
        assert oracle_mod.solve(g, mode, B, "mc").t_star == sum(g.T)
        rr = oracle_mod.solve(g, mode, B, "tc")
        assert rr.t_star >= sg.T(sg.sinks())
        assert oracle_mod.solve(g, mode, B + 1000, "tc").t_star == rr.t_star
        # below the budget floor there is no strategy
        assert oracle_mod.solve(g, mode, 2 * max(g.M) - 1).status == oracle_mod.INFEASIBLE


@pytest.mark.parametrize("name,make", GRAPHS)
def test_monotone_in_budget_and_family(oracle_mod, name, make):
    g = make()
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    budgets = sorted({lo - 1, lo, lo + (hi - lo) // 6, lo + (hi - lo) // 3, (lo + hi) // 2, hi})
    prev = {}
    exact_tables = {}
    for B in budgets:
        for mode in ("exact", "pruned"):
            r = oracle_mod.solve(g, mode, B, "tc")
            opt = INF_as_big(r.table()[0])
            if mode in prev:
                pB, popt, pts = prev[mode]
                assert np.all(opt <= popt)                  # pointwise in B
                if pts is not None:
                    assert r.t_star != -1 and r.t_star <= pts
            prev[mode] = (B, opt, r.t_star if r.status == oracle_mod.OK else None)
            sets = [tuple(row) for row in r.sets()]
            if mode == "exact":
                exact_tables[B] = (sets, opt, r.t_star, r.status)
            else:
                esets, eopt, ets, est = exact_tables[B]
                index = {s: i for i, s in enumerate(esets)}
                for i, s in enumerate(sets):
                    assert np.all(opt[i] >= eopt[index[s]])   # pruned >= exact
                if r.status == oracle_mod.OK:
                    assert est == oracle_mod.OK and r.t_star >= ets


@pytest.mark.parametrize("name,make", GRAPHS)
def test_row_minimum_is_t_free_dp(oracle_mod, name, make):
    g = make()
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for B in (lo, (2 * lo + hi) // 3, hi):
        for mode in ("exact", "pruned"):
            f, F = t_free_min_cache(g, mode, B)
            r = oracle_mod.solve(g, mode, B, "tc")
            opt = r.table()[0]
            for i in range(len(F)):
                row = opt[i][opt[i] >= 0]
                assert (row.min() if row.size else None) == f[i]


@pytest.mark.parametrize("name,make", GRAPHS)
def test_support_bound(oracle_mod, name, make):
    g = make()
    sg = bf.SetGraph(g)
    r = oracle_mod.solve(g, "exact", 2 * sum(g.M) // 2, "tc")
    opt = r.table()[0]
    for i, row in enumerate(r.sets()):
        L = sum(1 << v for v in range(g.n) if row[v])
        w = sg.T(L & ~sg.boundary(L))
        assert np.all(opt[i, w + 1:] == -1)
    finite = np.nonzero(opt[-1] >= 0)[0]
    assert finite.size == 0 or finite.min() >= sg.T(sg.sinks())
