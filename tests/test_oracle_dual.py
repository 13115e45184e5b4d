"""Pin the memory-indexed oracle (oracle/dual.py) to Algorithm 1.

The dual keeps, per (lower set, cached memory m), the least (time-centric)
or greatest (memory-centric) forward time t; its optimum must be Algorithm
1's t* with m* = opt[V, t*].  Checked against the C oracle (Algorithm 1 as
printed, itself pinned by brute force) on random DAGs, both families, both
objectives and budgets from 0 to unconstrained, and directly against brute
force over every chain (the naive search of Section 4.1) on tiny graphs.
"""

import pytest

from oracle import dual
from paper_1905_11722_amd import workloads as W
from tests import bruteforce as bf

BUDGETS = (0, 8, 20, 35, 60, 1000)


def _alg1(O, g, mode, B, objective):
    r = O.solve(g, mode, B, objective)
    assert r.status in (O.OK, O.INFEASIBLE)
    return (r.t_star, r.m_star) if r.t_star >= 0 else (None, None)


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("mode", ["exact", "pruned"])
def test_random_dags_match_algorithm1(oracle_mod, seed, mode):
    g = W.random_dag(9, 0.35, seed)
    for objective in ("tc", "mc"):
        for B in BUDGETS:
            d = dual.solve(g, mode, B, objective)
            assert (d["t"], d["m"]) == _alg1(oracle_mod, g, mode, B, objective), (seed, mode, objective, B)


@pytest.mark.parametrize("name", ["chain16", "layered24", "ladder40", "resnet50_t10", "unet_t10"])
def test_workloads_match_algorithm1(oracle_mod, name):
    c = W.case(name)
    for objective in ("tc", "mc"):
        d = dual.solve(c.graph, c.mode, c.B, objective)
        assert (d["t"], d["m"]) == _alg1(oracle_mod, c.graph, c.mode, c.B, objective), (name, objective)


@pytest.mark.parametrize("seed", range(6))
def test_brute_force(seed):
    g = W.random_dag(6, 0.4, seed)
    for mode in ("exact", "pruned"):
        for B in (6, 15, 30, 200):
            F, opt, _ = bf.brute_table(g, mode, B)
            for objective in ("tc", "mc"):
                t = bf.select(opt, F, objective)
                d = dual.solve(g, mode, B, objective)
                if t is None:
                    assert d["t"] is None
                else:
                    assert (d["t"], d["m"]) == (t, opt[(len(F) - 1, t)]), (seed, mode, B, objective)


def test_degenerate_graphs(oracle_mod):
    # one node: the only chain is {} -> {v}; v has no successor, so its
    # boundary is empty (t = T_v, nothing cached, m = 0) and the segment
    # needs 2 M_v
    g = W.Graph(n=1, succ=[[]], T=[3], M=[5])
    for mode in ("exact", "pruned"):
        assert dual.solve(g, mode, 9, "tc")["t"] is None
        d = dual.solve(g, mode, 10, "tc")
        assert (d["t"], d["m"]) == (3, 0)
    # an antichain: no node has a successor, so no chain caches anything and
    # every chain repeats the whole forward time
    g = W.antichain(5, seed=1)
    for objective in ("tc", "mc"):
        d = dual.solve(g, "exact", 10_000, objective)
        assert (d["t"], d["m"]) == (sum(g.T), 0)
        assert (d["t"], d["m"]) == _alg1(oracle_mod, g, "exact", 10_000, objective)


def test_work_is_the_budget_window():
    """Each pair relaxes the m with m + c <= B inside the row: never more
    than pairs * (min(B, M(V)) + 1)."""
    c = W.case("ladder40")
    d = dual.solve(c.graph, c.mode, c.B, "tc")
    assert 0 < d["relaxations"] <= d["pairs"] * d["width"]
    assert d["width"] == min(c.B, sum(c.graph.M)) + 1


MUTANTS = [
    ("top = min(B - c, width - 1 - dM)", "top = min(B, width - 1 - dM)"),          # no budget test
    ("c = 2 * M[Vp].sum() + out[j]", "c = M[Vp].sum() + out[j]"),                  # Eq. 2 term (ii) once
    ("c = 2 * M[Vp].sum() + out[j]", "c = 2 * M[Vp].sum()"),                       # terms (iii), (iv) dropped
    ("dT = T[Vp & ~bd[j]].sum()", "dT = T[Vp].sum()"),                            # boundary not excluded
    ("dM = M[bd[j] & ~L].sum()", "dM = M[bd[j]].sum()"),                          # boundary counted twice
    ("out[j] = M[dp & ~L].sum() + M[dmdp & ~L].sum()", "out[j] = M[dp & ~L].sum()"),
    ("m = int(np.flatnonzero(row == t)[0])", "m = int(np.flatnonzero(row == t)[-1])"),
    ("np.maximum(dst, cand, out=dst)", "np.minimum(dst, np.where(cand < 0, INF, cand), out=dst)"),
]


@pytest.mark.parametrize("k", range(len(MUTANTS)))
def test_planted_mistakes_are_caught(oracle_mod, k):
    """Each plausible mistake, planted in a copy of the dual oracle on the
    CPU, makes at least one of the comparisons above fail."""
    import inspect
    import types
    src = inspect.getsource(dual)
    a, b = MUTANTS[k]
    assert src.count(a) == 1
    mod = types.ModuleType("dual_mutant")
    exec(compile(src.replace(a, b), "dual_mutant", "exec"), mod.__dict__)
    caught = False
    for seed in range(12):
        g = W.random_dag(9, 0.35, seed)
        for mode in ("exact", "pruned"):
            for objective in ("tc", "mc"):
                for B in BUDGETS:
                    try:
                        got = mod.solve(g, mode, B, objective)
                        got = (got["t"], got["m"])
                    except Exception:
                        caught = True
                        break
                    if got != _alg1(oracle_mod, g, mode, B, objective):
                        caught = True
                        break
                if caught:
                    break
            if caught:
                break
        if caught:
            break
    assert caught, MUTANTS[k]
