"""The unit of work behind every relaxations/s figure, pinned on the CPU.

tests/family_stats.py counts, from the oracle's family with plain set
operations, the pairs (L, L'), the table cells sum w_L and the relaxations
sum over pairs of w_L, with w_L = T(L \\ boundary(L)) + 1.  Pins:
 - w_L is exactly the support of row L in Algorithm 1's table (Appendix A):
   at B = 2 M(V) every chain fits the budget, the chain (empty, L) reaches
   t = T(L \\ boundary(L)), and no chain ending at L goes further, so the last
   finite cell of row L in the oracle's table sits at w_L - 1;
 - the pair count equals the pairs the oracle's fill loop visits;
 - closed forms of chains (prefix family) and antichains (all subsets);
 - the stored values of the benchmark workloads (golden/family_stats.json,
   written by golden/make_family_stats.py) are what the counter gives today.
"""

import json
import os

import numpy as np
import pytest

from oracle import oracle as O
from paper_1905_11722_amd import workloads as W
from tests.family_stats import family_stats

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "family_stats.json")


def support_matches(g, mode):
    s = family_stats(g, mode)
    ref = O.solve(g, mode, 2 * sum(g.M), "tc", parallel=True)
    assert ref.status == O.OK
    assert ref.num_sets == s["num_sets"]
    assert ref.num_pairs == s["num_pairs"]
    opt, _ = ref.table()
    last = np.array([np.nonzero(row >= 0)[0].max() for row in opt])
    np.testing.assert_array_equal(last + 1, s["w"])
    return s


@pytest.mark.parametrize("name", ["chain16", "layered24", "ladder40", "unet_t10",
                                  "resnet50_t10", "densenet121_t10"])
def test_support_is_row_width(name):
    c = W.case(name)
    for mode in ("exact", "pruned") if c.mode == "exact" else ("pruned",):
        support_matches(c.graph, mode)


@pytest.mark.parametrize("seed", range(10))
def test_support_random_dags(seed):
    g = W.random_dag(9, 0.3, 400 + seed, tmax=30, mmax=9)
    for mode in ("exact", "pruned"):
        support_matches(g, mode)


def test_chain_closed_form():
    g = W.chain(12, seed=5, tmax=9, mmax=7)
    n, T = g.n, np.array(g.T)
    s = family_stats(g, "exact")
    # prefixes L_k = {0..k-1}: boundary {k-1} for 0 < k < n, empty for k = 0, n
    w = [1] + [int(T[:k - 1].sum()) + 1 for k in range(1, n)] + [int(T.sum()) + 1]
    assert s["num_sets"] == n + 1
    assert s["num_pairs"] == (n + 1) * n // 2
    assert s["table_cells"] == sum(w)
    assert s["relaxations"] == sum(w[k] * (n - k) for k in range(n + 1))


def test_antichain_closed_form():
    g = W.antichain(6, seed=2, tmax=9, mmax=7)
    s = family_stats(g, "exact")
    # every subset is a lower set with an empty boundary (no node has a
    # successor), so w_L = T(L) + 1; each node lies in half of the 2^n
    # subsets, and L is a proper subset of 2^(n - |L|) - 1 others
    n, T = g.n, np.array(g.T)
    assert s["num_sets"] == 2 ** n
    assert s["num_pairs"] == 3 ** n - 2 ** n
    assert s["table_cells"] == 2 ** n + 2 ** (n - 1) * int(T.sum())
    relax = 0
    for mask in range(2 ** n):
        members = [v for v in range(n) if mask >> v & 1]
        relax += (int(T[members].sum()) + 1) * (2 ** (n - len(members)) - 1)
    assert s["relaxations"] == relax


def test_golden_values_current():
    stored = json.load(open(GOLDEN))
    assert len(stored) == 9
    for name, want in stored.items():
        c = W.case(name)
        got = family_stats(c.graph, c.mode)
        for key in ("num_sets", "num_pairs", "table_cells", "relaxations", "max_row", "T_total"):
            assert got[key] == want[key], (name, key)
