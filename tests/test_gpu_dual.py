"""The memory-indexed table on the GPU (rc_solve_dual) versus the oracle.

rc_solve_dual must return exactly Algorithm 1's t* and opt[V, t*]: checked
against the memory-indexed oracle (oracle/dual.py, pinned to the C oracle
and to brute force) and against rc_solve on the same family, for both
objectives, both families, budgets from below the feasibility threshold to
unconstrained, and the degenerate graphs.  The chain traced back through the
table, its seg / cached and its Eq. 1 / Eq. 2 re-evaluation must equal the
oracle's bit for bit (same family order, same tie rule).
"""

import numpy as np

import pytest

from oracle import dual
from paper_1905_11722_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1905_11722_amd import rcdp
    rcdp.load_library()
    return rcdp


def _expect(d):
    return (-1, -1) if d["t"] is None else (d["t"], d["m"])


def check(rc, g, mode, budgets, objectives=("tc", "mc"), against_solve=True):
    fam = rc.Graph.create(g).build_family(mode)
    for B in budgets:
        for objective in objectives:
            d = dual.solve(g, mode, B, objective)
            t, m, ms = fam.solve_dual(B, objective)
            assert (t, m) == _expect(d), (mode, B, objective)
            t2, m2, _, sched = fam.solve_dual(B, objective, schedule=True)
            assert (t2, m2) == (t, m)
            if d["t"] is None:
                assert sched is None
            else:
                np.testing.assert_array_equal(sched.chain, d["chain"])
                np.testing.assert_array_equal(sched.seg, d["seg"])
                np.testing.assert_array_equal(sched.cached, d["cached"])
                assert (sched.overhead, sched.peak, sched.cache_mem) == (
                    d["overhead"], d["peak"], d["cache_mem"])
                assert (sched.overhead, sched.cache_mem) == (t, m) and sched.peak <= B
            if against_solve and B <= 60000:
                sol = fam.solve(B, objective)
                assert (t, m) == (sol.t_star, sol.m_star), (mode, B, objective)
                sol.free()


@pytest.mark.parametrize("name", list(W.CASES))
def test_workloads(rc, name):
    c = W.case(name)
    check(rc, c.graph, c.mode, [c.B])


RANDOM = [(n, p, seed) for seed, (n, p) in enumerate(
    [(n, p) for n in (3, 5, 7, 9, 11) for p in (0.2, 0.5, 0.8)])]


@pytest.mark.parametrize("n,p,seed", RANDOM)
def test_random_dags(rc, n, p, seed):
    g = W.random_dag(n, p, 2000 + seed, tmax=40, mmax=30)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    budgets = (0, lo - 1, lo, (2 * lo + hi) // 3, (lo + hi) // 2, hi, 10 ** 7)
    for mode in ("exact", "pruned"):
        check(rc, g, mode, budgets)


def test_wide_memory_rows(rc):
    """Rows of many 256-cell tiles (M(V) in the thousands) and a ragged tail."""
    g = W.random_dag(14, 0.3, 77, tmax=20, mmax=700)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    check(rc, g, "pruned", (lo, (lo + hi) // 2, hi - 1, hi))
    check(rc, g, "exact", ((lo + hi) // 2,))


def test_empty_and_single(rc):
    g0 = W.Graph(0, [], [], [])
    for mode in ("exact", "pruned"):
        fam = rc.Graph.create(g0).build_family(mode)
        assert fam.solve_dual(0, "tc")[:2] == (0, 0)
        assert fam.solve_dual(5, "mc")[:2] == (0, 0)
    g1 = W.chain(1, 3)
    for mode in ("exact", "pruned"):
        check(rc, g1, mode, (2 * g1.M[0] - 1, 2 * g1.M[0], 10 ** 6))


def test_bad_arguments_and_repeat(rc):
    c = W.case("ladder40")
    fam = rc.Graph.create(c.graph).build_family(c.mode)
    with pytest.raises(rc.RcError):
        fam.solve_dual(-1, "tc")
    with pytest.raises(rc.RcError):
        fam.solve_dual(c.B, 7)
    first = fam.solve_dual(c.B, "tc")[:2]
    for _ in range(3):
        assert fam.solve_dual(c.B, "tc")[:2] == first


def test_wide_levels_exact_antichain(rc):
    """An antichain of 15 nodes: the exact family is all 2^15 subsets, with
    size levels of up to 6435 targets and targets of up to 32767 pairs (many
    blocks along y and z).  Against rc_solve on the same family (the oracle
    is too slow here) and by re-evaluating the schedule."""
    g = W.antichain(15, seed=3)
    fam = rc.Graph.create(g).build_family("exact")
    assert fam.info["num_sets"] == 1 << 15
    for B in (2 * max(g.M), sum(g.M), 2 * sum(g.M)):
        for objective in ("tc", "mc"):
            t, m, _, sched = fam.solve_dual(B, objective, schedule=True)
            sol = fam.solve(B, objective)
            assert (t, m) == (sol.t_star, sol.m_star), (B, objective)
            sol.free()
            assert (sched.overhead, sched.cache_mem) == (t, m) and sched.peak <= B


def test_node_limit(rc):
    """4096 nodes: the memory-indexed solve of a unit-cost chain (4097 sets,
    a 4096-step traceback) and of an antichain, against the closed forms
    pinned in test_oracle_closed.py: the chain's least overhead 1 with n - 1
    cached nodes and every prefix as the chain, its memory-centric optimum
    the one-segment chain; the antichain's T(V) at no cached memory."""
    from tests.closed_forms import antichain_pruned_expected
    n = 4096
    g = W.Graph(n, [[v + 1] if v + 1 < n else [] for v in range(n)], [1] * n, [1] * n)
    fam = rc.Graph.create(g).build_family("pruned")
    t, m, _, sched = fam.solve_dual(2 * n, "tc", schedule=True)
    assert (t, m) == (1, n - 1)
    assert sched.chain.tolist() == list(range(1, n + 1))
    assert (sched.overhead, sched.peak, sched.cache_mem) == (1, n + 1, n - 1)
    t, m, _, sched = fam.solve_dual(2 * n, "mc", schedule=True)
    assert (t, m) == (n, 0) and sched.chain.tolist() == [n]
    g = W.antichain(n, seed=5, tmax=1, mmax=5)
    fam = rc.Graph.create(g).build_family("pruned")
    MV, big = sum(g.M), max(g.M)
    for B in (2 * MV, 2 * (MV - big), 2 * (MV - big) - 1):
        _, _, chain = antichain_pruned_expected(g, B)
        t, m, _, sched = fam.solve_dual(B, "tc", schedule=True)
        if chain is None:
            assert (t, m) == (-1, -1)
        else:
            assert (t, m) == (sum(g.T), 0)
            assert sched.overhead == sum(g.T) and sched.cache_mem == 0 and sched.peak <= B
