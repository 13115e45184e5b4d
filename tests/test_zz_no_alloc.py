"""rc_solve_dual_noalloc (the memory-indexed solve in the library's static
scratch, for callers that cannot allocate) against rc_solve_dual on the same
family: t*, opt[V, t*], the traced chain, seg, cached and the Eq. 1 / Eq. 2
re-evaluation, bit for bit, on consecutive calls that share the scratch --
a large solve, then a smaller one, then the large one again -- and the
clear error for a solve that needs more than the scratch."""

import numpy as np
import pytest

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


def same(a, b):
    ta, ma, fa, sa = a
    tb, mb, sb = b
    assert (ta, ma) == (tb, mb)
    if sa is None:
        assert sb is None
        return
    np.testing.assert_array_equal(sa.chain, sb.chain)
    np.testing.assert_array_equal(sa.seg, sb.seg)
    np.testing.assert_array_equal(sa.cached, sb.cached)
    assert (sa.overhead, sa.peak, sa.cache_mem) == (sb.overhead, sb.peak, sb.cache_mem)


def check(fam, B, objective):
    ref = fam.solve_dual(B, objective, schedule=True)
    got = fam.solve_dual_noalloc(B, objective)
    same(ref, got)
    return got


def test_consecutive_calls_share_the_scratch(rc):
    big = W.case("densenet121")
    small = W.case("chain16")
    fb = rc.Graph.create(big.graph).build_family(big.mode)
    fs = rc.Graph.create(small.graph).build_family(small.mode)
    for objective in ("tc", "mc"):
        first = check(fb, big.B, objective)              # large table
        check(fs, small.B, objective)                    # smaller input, same scratch
        again = check(fb, big.B, objective)
        assert first[:2] == again[:2]
    check(fs, 2 * max(small.graph.M) - 1, "tc")          # infeasible
    check(fs, 0, "mc")


@pytest.mark.parametrize("name", ["unet", "resnet50", "ladder40", "layered24"])
def test_workloads(rc, name):
    c = W.case(name)
    fam = rc.Graph.create(c.graph).build_family(c.mode)
    for B in (c.B, fam.min_budget(), 2 * sum(c.graph.M)):
        for objective in ("tc", "mc"):
            check(fam, B, objective)


def test_too_large_for_the_scratch(rc):
    g = W.antichain(12, seed=3, tmax=5, mmax=900)         # 4096 sets, rows of M(V) + 1
    fam = rc.Graph.create(g).build_family("exact")
    B = 2 * sum(g.M)
    assert fam.info["num_sets"] * (sum(g.M) + 1) * 4 > 16 << 20
    with pytest.raises(rc.RcError) as e:
        fam.solve_dual_noalloc(B, "tc")
    assert e.value.status == rc.E_SCRATCH
    t, m, _ = fam.solve_dual(B, "tc")                     # the allocating path still works
    assert t >= 0
