"""The dominance skip on the GPU (rc_solve_dominance) versus the oracle.

The oracle runs Algorithm 1 with the skip of Section 4.2's last paragraph
(oracle_solve_dominance, pinned to brute force).  The GPU keeps of each row
its weak front only (the cells no earlier cell of the row beats on memory)
and stores infinity elsewhere, so its table must equal the oracle's skipped
table with that same front taken row by row, bit for bit; the optarg of every
front cell, t*, opt[V, t*] and the traced schedule (same tie rule) must equal
the oracle's.  The full-size ResNet-50, DenseNet-121 and U-Net shapes run the
same comparison against the oracle's all-cores build (identical results,
pinned in test_oracle_parallel.py).
"""

import numpy as np
import pytest

from oracle import oracle as O
from paper_1905_11722_amd import workloads as W
from tests.trace_paths import reconstruct_each

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1905_11722_amd import rcdp
    rcdp.load_library()
    return rcdp


def front(rows):
    """Keep, per row, the finite cells no larger than every earlier finite
    cell (-1 = infinite)."""
    inf = np.iinfo(np.int64).max
    x = np.where(rows < 0, inf, rows)
    earlier = np.minimum.accumulate(np.concatenate([np.full((x.shape[0], 1), inf), x[:, :-1]], 1), 1)
    keep = (rows >= 0) & (x <= earlier)
    return np.where(keep, rows, -1), keep


def compare(rc, g, mode, B, parallel=False):
    fam = rc.Graph.create(g).build_family(mode)
    ref = O.solve_dominance(g, mode, B, parallel=parallel)
    assert ref.status in (O.OK, O.INFEASIBLE)
    sol = fam.solve_dominance(B)
    full = fam.solve(B, "tc")
    assert (sol.t_star, sol.m_star) == (full.t_star, full.m_star)
    if ref.status == O.INFEASIBLE:
        assert sol.status == rc.INFEASIBLE and (sol.t_star, sol.m_star) == (-1, -1)
    else:
        assert (sol.t_star, sol.m_star) == (ref.t_star, ref.m_star)
        chain, seg, cached = ref.schedule()
        for sched in reconstruct_each(sol, ref.num_sets):
            np.testing.assert_array_equal(sched.chain, chain)
            np.testing.assert_array_equal(sched.seg, seg)
            np.testing.assert_array_equal(sched.cached, cached)
            assert (sched.overhead, sched.peak, sched.cache_mem) == (
                ref.overhead, ref.peak, ref.cache_mem)
    m, a = sol.table()
    rm, ra = ref.table()
    want, keep = front(rm)
    np.testing.assert_array_equal(m, want)
    np.testing.assert_array_equal(a[keep], ra[keep])
    np.testing.assert_array_equal(front(full.table()[0])[0], m)   # fronts are kept
    sol.free()
    full.free()


@pytest.mark.parametrize("name", ["chain16", "layered24", "ladder40", "unet_t10", "resnet50_t10"])
def test_workloads(rc, name):
    c = W.case(name)
    g = c.graph
    for B in (c.B, 2 * max(g.M), 2 * sum(g.M)):
        compare(rc, g, c.mode, B)


@pytest.mark.parametrize("seed", range(8))
def test_random_dags(rc, seed):
    g = W.random_dag(9, 0.35, 300 + seed, tmax=40, mmax=12)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for mode in ("exact", "pruned"):
        for B in (0, lo - 1, lo, (lo + hi) // 2, hi):
            compare(rc, g, mode, B)


def test_rows_of_several_tiles(rc):
    """Rows of a few thousand cells: several 1024-cell tiles of the level
    fill and 256-cell chunks of the front pass, with a ragged tail."""
    g = W.random_dag(13, 0.3, 41, tmax=400, mmax=30)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for B in (lo, (lo + hi) // 2, hi):
        compare(rc, g, "pruned", B)
    compare(rc, g, "exact", (lo + hi) // 2)


def test_degenerate(rc):
    for mode in ("exact", "pruned"):
        fam = rc.Graph.create(W.Graph(0, [], [], [])).build_family(mode)
        s = fam.solve_dominance(0)
        assert (s.t_star, s.m_star) == (0, 0)
    g1 = W.chain(1, 3)
    for mode in ("exact", "pruned"):
        for B in (2 * g1.M[0] - 1, 2 * g1.M[0]):
            compare(rc, g1, mode, B)
    with pytest.raises(rc.RcError):
        rc.Graph.create(g1).build_family("exact").solve_dominance(-1)


@pytest.mark.slow
@pytest.mark.parametrize("name", ["resnet50", "unet", "densenet121"])
def test_full_size_against_oracle(rc, name):
    """The whole skipped table (every row's front), the optarg of every front
    cell, t*, opt[V, t*] and the schedule against the oracle with the skip."""
    c = W.case(name)
    compare(rc, c.graph, c.mode, c.B, parallel=True)
