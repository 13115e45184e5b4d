"""Pin the oracle's whole table against brute force over every chain.

Brute force is the paper's own naive exhaustive search (Section 4.1),
written separately from the oracle in tests/bruteforce.py.  The checks
cover opt[L, t] for every family member and every t in 0..T(V), optarg
(smallest penultimate family index among optimal chains), t* for both
objectives (Section 4.2 and 4.4), feasibility, and the returned schedule.
"""

import numpy as np
import pytest

from paper_1905_11722_amd import workloads as W
from tests import bruteforce as bf


def _check_against_brute(O, g, mode, B):
    F, bopt, barg = bf.brute_table(g, mode, B)
    r = O.solve(g, mode, B, "tc")
    assert r.status in (O.OK, O.INFEASIBLE)
    sets = r.sets()
    # family: same members in the same order
    fam = [sum(1 << v for v in range(g.n) if row[v]) for row in sets]
    assert fam == F
    opt, arg = r.table()
    TV = sum(g.T)
    exp_opt = np.full((len(F), TV + 1), -1, dtype=np.int64)
    exp_arg = np.full((len(F), TV + 1), -1, dtype=np.int32)
    for (i, t), m in bopt.items():
        exp_opt[i, t] = m
        exp_arg[i, t] = barg[(i, t)]
    np.testing.assert_array_equal(opt, exp_opt)
    np.testing.assert_array_equal(arg, exp_arg)
    for objective in ("tc", "mc"):
        ts = bf.select(bopt, F, objective)
        ro = O.solve(g, mode, B, objective)
        if ts is None:
            assert ro.status == O.INFEASIBLE
            continue
        assert ro.status == O.OK
        assert ro.t_star == ts
        assert ro.m_star == bopt[(len(F) - 1, ts)]
        # returned chain: ends at V, re-evaluates to t* with peak <= B
        chain, seg, cached = ro.schedule()
        assert chain[-1] == len(F) - 1
        sg = bf.SetGraph(g)
        ovh, peak, mu = bf.evaluate_chain(sg, [F[c] for c in chain])
        assert (ovh, peak, mu) == (ro.overhead, ro.peak, ro.cache_mem)
        assert ovh == ts and peak <= B and mu == ro.m_star
    return r


def _budgets(g):
    M = g.M
    lo = 2 * max(M)
    hi = 2 * sum(M)
    return sorted({lo - 1, lo, (lo + hi) // 3, (lo + hi) // 2, hi, hi + 5})


CASES = []
for seed in range(12):
    n = 3 + seed % 5                          # 3..7 nodes, any density
    p = [0.15, 0.35, 0.6][seed % 3]
    CASES.append((n, p, seed))
for seed in range(100, 106):
    CASES.append((9, 0.45, seed))             # denser, 9 nodes


@pytest.mark.parametrize("n,p,seed", CASES)
@pytest.mark.parametrize("mode", ["exact", "pruned"])
def test_random_dag_tables(oracle_mod, n, p, seed, mode):
    g = W.random_dag(n, p, seed, tmax=9, mmax=7)
    for B in _budgets(g):
        _check_against_brute(oracle_mod, g, mode, B)


@pytest.mark.parametrize("mode", ["exact", "pruned"])
def test_antichain6(oracle_mod, mode):
    g = W.antichain(6, seed=3)
    for B in _budgets(g):
        _check_against_brute(oracle_mod, g, mode, B)


@pytest.mark.parametrize("seed", range(4))
def test_small_ladder(oracle_mod, seed):
    g = W.ladder(4, seed=seed, tmax=9, mmax=9)
    for B in _budgets(g):
        _check_against_brute(oracle_mod, g, "exact", B)


def test_layered_small(oracle_mod):
    g = W.layered(3, 3, seed=5, tmax=20, mmax=12)
    for B in _budgets(g):
        _check_against_brute(oracle_mod, g, "exact", B)
        _check_against_brute(oracle_mod, g, "pruned", B)


def test_single_node(oracle_mod):
    g = W.chain(1, 0)
    r = _check_against_brute(oracle_mod, g, "exact", 2 * g.M[0])
    assert r.t_star == g.T[0]
    r = oracle_mod.solve(g, "exact", 2 * g.M[0] - 1)
    assert r.status == oracle_mod.INFEASIBLE


def test_empty_graph(oracle_mod):
    g = W.Graph(0, [], [], [])
    r = oracle_mod.solve(g, "exact", 0)
    assert r.status == oracle_mod.OK
    assert (r.num_sets, r.T_total, r.t_star, r.m_star, r.k) == (1, 0, 0, 0, 0)
    r = oracle_mod.solve(g, "pruned", 0)
    assert (r.num_sets, r.t_star, r.k) == (1, 0, 0)


@pytest.mark.parametrize("n,p,seed", CASES[:12])
@pytest.mark.parametrize("mode", ["exact", "pruned"])
def test_min_budget(oracle_mod, n, p, seed, mode):
    """The oracle's bisection for the smallest feasible budget (Section 5)
    against the least peak over every chain."""
    g = W.random_dag(n, p, seed, tmax=9, mmax=7)
    b = oracle_mod.min_budget(g, mode)
    assert b == bf.brute_min_budget(g, mode)
    assert b >= 2 * max(g.M)                       # every node lies in a segment
    assert oracle_mod.solve(g, mode, b, "tc").status == oracle_mod.OK
    assert oracle_mod.solve(g, mode, b - 1, "tc").status == oracle_mod.INFEASIBLE
