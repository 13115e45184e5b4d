"""Closed forms that pin the oracle (no DP involved on the checking side).

* Chains: the lower sets of a chain are its prefixes, so a strategy is a
  set of cut points.  Eq. 1 and Eq. 2 then reduce to sums over the cuts
  (term (iv) of Eq. 2 is empty and term (iii) is the node after the cut);
  every cut set is enumerated directly.
* Family sizes of graphs whose lower sets can be counted by hand
  (Section 2 bounds: #V <= #L_G <= 2^#V, counting the empty set).
"""

import itertools

import numpy as np
import pytest

from paper_1905_11722_amd import workloads as W


def chain_strategies(T, M):
    """Yield (overhead, peak, cache) for every cut set of a chain."""
    n = len(T)
    for r in range(n):
        for cuts in itertools.combinations(range(1, n), r):
            ends = list(cuts) + [n]
            start = 0
            cached = 0
            peak = 0
            for e in ends:
                seg = 2 * sum(M[start:e])
                nxt = M[e] if e < n else 0
                peak = max(peak, cached + seg + nxt)
                if e < n:
                    cached += M[e - 1]     # the last node of the prefix stays
                start = e
            overhead = sum(T) - sum(T[c - 1] for c in cuts)
            yield overhead, peak, cached


def chain_row_V(T, M, B):
    best = {}
    for ovh, peak, cache in chain_strategies(T, M):
        if peak <= B and (ovh not in best or cache < best[ovh]):
            best[ovh] = cache
    return best


@pytest.mark.parametrize("n,seed", [(2, 1), (5, 2), (8, 3), (11, 4), (13, 5)])
def test_chain_row_V_closed_form(oracle_mod, n, seed):
    g = W.chain(n, seed)
    for B in range(2 * max(g.M) - 1, 2 * sum(g.M) + 2, max(1, sum(g.M) // 7)):
        best = chain_row_V(g.T, g.M, B)
        for mode in ("exact", "pruned"):
            r = oracle_mod.solve(g, mode, B, "tc")
            opt, _ = r.rows(r.num_sets - 1, 1)
            exp = np.full(sum(g.T) + 1, -1, dtype=np.int64)
            for t, m in best.items():
                exp[t] = m
            np.testing.assert_array_equal(opt[0], exp)
            if best:
                assert r.t_star == min(best)
                assert oracle_mod.solve(g, mode, B, "mc").t_star == max(best)
            else:
                assert r.status == oracle_mod.INFEASIBLE


def test_chain16_at_64(oracle_mod):
    """The 16-node chain at B = 64: all 2^15 cut sets by the closed form."""
    c = W.case("chain16")
    g = c.graph
    best = chain_row_V(g.T, g.M, c.B)
    r = oracle_mod.solve(g, "exact", c.B, "tc")
    assert r.t_star == min(best) == 21
    assert r.m_star == best[21] == 47
    assert oracle_mod.solve(g, "exact", c.B, "mc").t_star == max(best) == 92
    bmin = min(peak for _, peak, _ in chain_strategies(g.T, g.M))
    assert bmin == 45
    assert oracle_mod.min_budget(g, "exact") == bmin
    assert oracle_mod.solve(g, "exact", bmin, "tc").status == oracle_mod.OK
    assert oracle_mod.solve(g, "exact", bmin - 1, "tc").status == oracle_mod.INFEASIBLE


@pytest.mark.parametrize("n", [1, 4, 9])
def test_family_sizes_chain(oracle_mod, n):
    g = W.chain(n, 0)
    for mode in ("exact", "pruned"):
        assert oracle_mod.solve(g, mode, 10 ** 6).num_sets == n + 1


@pytest.mark.parametrize("n", [1, 3, 6])
def test_family_sizes_antichain(oracle_mod, n):
    g = W.antichain(n)
    assert oracle_mod.solve(g, "exact", 10 ** 6).num_sets == 2 ** n
    # singletons, the empty set, and V (which is a singleton when n == 1)
    assert oracle_mod.solve(g, "pruned", 10 ** 6).num_sets == n + 1 + (n > 1)


@pytest.mark.parametrize("a,b", [(3, 4), (5, 2), (6, 6)])
def test_family_sizes_two_chains(oracle_mod, a, b):
    succ = [[v + 1] if v + 1 < a else [] for v in range(a)]
    succ += [[a + v + 1] if v + 1 < b else [] for v in range(b)]
    g = W.Graph(a + b, succ, [1] * (a + b), [1] * (a + b))
    assert oracle_mod.solve(g, "exact", 10 ** 6).num_sets == (a + 1) * (b + 1)


def test_family_size_ladder_cross_every_node(oracle_mod):
    """Ladder with a cross edge a_i -> b_i at every i: a lower set takes a
    prefix of a of length p and a prefix of b of length q <= p, so there are
    (L+1)(L+2)/2 of them."""
    L = 6
    g = W.ladder(L, seed=0, cross_every=1)
    assert oracle_mod.solve(g, "exact", 10 ** 6).num_sets == (L + 1) * (L + 2) // 2


def test_family_exceeds_cap(oracle_mod):
    g = W.antichain(8)
    r = oracle_mod.solve(g, "exact", 10 ** 6, max_sets=255)
    assert r.status == oracle_mod.E_TOO_MANY_SETS
    assert oracle_mod.solve(g, "exact", 10 ** 6, max_sets=256).num_sets == 256


@pytest.mark.parametrize("n,seed", [(2, 0), (5, 1), (12, 2), (30, 3)])
def test_antichain_pruned_closed_form(oracle_mod, n, seed):
    """The closed form the GPU tests use at the node limit (pruned family of
    an antichain: every boundary empty, nothing cached, the one-segment chain
    or empty -> {v} -> V) equals the oracle's whole table and traced chain at
    the unconstrained budget, at one where only a two-segment chain fits, and
    at an infeasible one."""
    from tests.closed_forms import antichain_pruned_expected
    g = W.antichain(n, seed=seed, tmax=3, mmax=5)
    MV, big = sum(g.M), max(g.M)
    budgets = [2 * MV, 2 * (MV - big), 2 * (MV - big) - 1, 2 * big - 1]
    for B in [b for b in budgets if b >= 0]:
        em, ea, chain = antichain_pruned_expected(g, B)
        r = oracle_mod.solve(g, "pruned", B, "tc")
        m, a = r.table()
        np.testing.assert_array_equal(m, em, err_msg=f"n={n} B={B}")
        np.testing.assert_array_equal(a, ea, err_msg=f"n={n} B={B}")
        if chain is None:
            assert r.status == oracle_mod.INFEASIBLE
        else:
            assert list(r.schedule()[0]) == chain


@pytest.mark.parametrize("n", [2, 5, 8, 20])
def test_unit_chain_closed_form(oracle_mod, n):
    """The closed form the GPU tests use for a 4096-node chain with unit
    costs at an unconstrained budget: least overhead 1 with every node but
    the sink cached (all n prefixes as the chain, peak n + 1), row V
    opt[V, t] = n - t for t >= 1, and the memory-centric optimum the
    one-segment chain (t = n, m = 0, peak 2 n)."""
    g = W.Graph(n, [[v + 1] if v + 1 < n else [] for v in range(n)], [1] * n, [1] * n)
    r = oracle_mod.solve(g, "pruned", 2 * n, "tc")
    assert (r.num_sets, r.num_pairs) == (n + 1, n * (n + 1) // 2)
    assert (r.t_star, r.m_star, r.overhead, r.peak, r.cache_mem) == (1, n - 1, 1, n + 1, n - 1)
    chain, seg, cached = r.schedule()
    assert list(chain) == list(range(1, n + 1)) and list(seg) == list(range(n))
    assert list(cached) == [True] * (n - 1) + [False]
    m, _ = r.table()
    assert m[n].tolist() == [-1] + [n - t for t in range(1, n + 1)]
    r = oracle_mod.solve(g, "pruned", 2 * n, "mc")
    assert (r.t_star, r.m_star, r.overhead, r.peak) == (n, 0, n, 2 * n)
    assert list(r.schedule()[0]) == [n]
