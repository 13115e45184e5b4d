"""rc_family_stats against the CPU count of the DP's unit of work.

The relaxation count (sum over pairs (L, L') of w_L, w_L = T(L \\ boundary(L))
+ 1) divides every relaxations/s figure the benchmark reports, and the table
cells size the table.  The library computes both on the device while it
builds the family; here they are compared with the count from the oracle's
family (tests/family_stats.py, pinned in test_family_stats.py): the stored
values of the nine benchmark workloads and a direct count on random DAGs.
"""

import json
import os

import pytest

from paper_1905_11722_amd import workloads as W
from tests.family_stats import family_stats

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "family_stats.json")
KEYS = ("num_sets", "num_pairs", "table_cells", "relaxations", "max_row", "T_total")


@pytest.fixture(scope="module")
def rc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1905_11722_amd import rcdp
    rcdp.load_library()
    return rcdp


@pytest.mark.parametrize("name", sorted(json.load(open(GOLDEN))))
def test_workloads(rc, name):
    want = json.load(open(GOLDEN))[name]
    c = W.case(name)
    info = rc.Graph.create(c.graph).build_family(c.mode).info
    for key in KEYS:
        assert info[key] == want[key], (name, key)


@pytest.mark.parametrize("seed", range(8))
def test_random_dags(rc, seed):
    g = W.random_dag(11, 0.3, 600 + seed, tmax=200, mmax=20)
    for mode in ("exact", "pruned"):
        want = family_stats(g, mode)
        info = rc.Graph.create(g).build_family(mode).info
        for key in KEYS:
            assert info[key] == want[key], (mode, key)
