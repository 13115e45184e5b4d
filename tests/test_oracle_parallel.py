"""The all-cores build of the oracle (OpenMP, the targets of one source split
among threads) returns exactly what the single-threaded build returns: the
whole opt / optarg table, t*, m*, the schedule and its re-evaluation, the
counts, with and without the dominance skip.  The benchmark's all-cores CPU
baseline and the full-size GPU parity tests run this build."""

import numpy as np
import pytest

from oracle import oracle as O
from paper_1905_11722_amd import workloads as W


def same(a, b):
    assert (a.status, a.num_sets, a.num_pairs, a.T_total, a.relaxations_literal) == (
        b.status, b.num_sets, b.num_pairs, b.T_total, b.relaxations_literal)
    assert (a.t_star, a.m_star, a.k, a.overhead, a.peak, a.cache_mem) == (
        b.t_star, b.m_star, b.k, b.overhead, b.peak, b.cache_mem)
    ma, aa = a.table()
    mb, ab = b.table()
    np.testing.assert_array_equal(ma, mb)
    np.testing.assert_array_equal(aa, ab)
    if a.status == O.OK:
        for x, y in zip(a.schedule(), b.schedule()):
            np.testing.assert_array_equal(x, y)


def test_parallel_build_has_threads():
    assert O.threads(parallel=False) == 1
    assert O.threads(parallel=True) >= 1


@pytest.mark.parametrize("name", ["chain16", "layered24", "ladder40", "unet_t10", "resnet50_t10"])
def test_workloads_identical(name):
    c = W.case(name)
    g = c.graph
    for B in (c.B, 2 * max(g.M), (c.B + 2 * sum(g.M)) // 2, 2 * sum(g.M)):
        for obj in ("tc", "mc"):
            same(O.solve(g, c.mode, B, obj), O.solve(g, c.mode, B, obj, parallel=True))
        same(O.solve_dominance(g, c.mode, B), O.solve_dominance(g, c.mode, B, parallel=True))


@pytest.mark.parametrize("seed", range(6))
def test_random_dags_identical(seed):
    g = W.random_dag(11, 0.3, 900 + seed, tmax=60, mmax=20)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for mode in ("exact", "pruned"):
        for B in (lo - 1, lo, (lo + hi) // 2, hi):
            same(O.solve(g, mode, B, "tc"), O.solve(g, mode, B, "tc", parallel=True))
    assert O.min_budget(g, "exact") == O.min_budget(g, "exact", parallel=True)
