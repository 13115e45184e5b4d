"""Input validation of the oracle (Section 2: G is a DAG, T_v, M_v > 0)."""

from paper_1905_11722_amd import workloads as W


def test_cycle(oracle_mod):
    g = W.Graph(3, [[1], [2], [0]], [1, 1, 1], [1, 1, 1])
    assert oracle_mod.solve(g, "exact", 10).status == oracle_mod.E_CYCLE
    g = W.Graph(2, [[0], []], [1, 1], [1, 1])        # self-loop
    assert oracle_mod.solve(g, "pruned", 10).status == oracle_mod.E_CYCLE


def test_nonpositive_costs(oracle_mod):
    g = W.chain(3, 0)
    assert oracle_mod.solve(g, "exact", 10, T=[1, 0, 1]).status == oracle_mod.E_COST
    assert oracle_mod.solve(g, "exact", 10, M=[1, 1, -2]).status == oracle_mod.E_COST


def test_bad_csr(oracle_mod):
    g = W.chain(3, 0)
    assert oracle_mod.solve(g, "exact", 10, csr=([0, 1, 2, 2], [1, 5])).status == oracle_mod.E_ARG
    assert oracle_mod.solve(g, "exact", 10, csr=([0, 2, 1, 2], [1, 2])).status == oracle_mod.E_ARG
    assert oracle_mod.solve(g, "exact", -1).status == oracle_mod.E_ARG


def test_duplicate_edges_collapse(oracle_mod):
    g = W.chain(4, 2)
    dup = ([0, 2, 3, 5, 5], [1, 1, 2, 3, 3])
    a = oracle_mod.solve(g, "exact", 30, csr=dup)
    b = oracle_mod.solve(g, "exact", 30)
    assert (a.status, a.t_star, a.m_star, a.num_sets) == (b.status, b.t_star, b.m_star, b.num_sets)
