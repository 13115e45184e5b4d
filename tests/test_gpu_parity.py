"""GPU path versus the oracle, bit for bit (all quantities are integers).

Every case runs the HIP library through its C ABI (rc_graph_create,
rc_build_family, rc_solve, rc_reconstruct, rc_export_table) and the C
oracle on the same seeded input, and compares: the family (members and
order), the whole opt / optarg table over t = 0..T(V), t* and opt[V, t*]
for both objectives, the traced chain, seg / cached, and the Eq. 1 / Eq. 2
re-evaluation of the schedule, from each traceback (predecessor scans,
optarg slice) forced in turn.
"""

import numpy as np
import pytest

from paper_1905_11722_amd import workloads as W

from tests.closed_forms import antichain_pruned_expected
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


def compare(rc, O, g, mode, B, objectives=("tc", "mc"), table=True, parallel=False):
    gg = rc.Graph.create(g)
    fam = gg.build_family(mode)
    ref = None
    for objective in objectives:
        ref = O.solve(g, mode, B, objective, parallel=parallel)
        assert ref.status in (O.OK, O.INFEASIBLE), ref.status
        sol = fam.solve(B, objective)
        assert fam.info["num_sets"] == ref.num_sets
        assert fam.info["num_pairs"] == ref.num_pairs
        assert fam.info["T_total"] == ref.T_total
        if ref.status == O.INFEASIBLE:
            assert sol.status == rc.INFEASIBLE
            assert (sol.t_star, sol.m_star) == (-1, -1)
        else:
            assert sol.status == rc.OK
            assert (sol.t_star, sol.m_star) == (ref.t_star, ref.m_star)
            chain, seg, cached = ref.schedule()
            for sched in reconstruct_each(sol, ref.num_sets):
                np.testing.assert_array_equal(sched.chain, chain)
                np.testing.assert_array_equal(sched.seg, seg)
                np.testing.assert_array_equal(sched.cached, cached)
                assert (sched.overhead, sched.peak, sched.cache_mem) == (
                    ref.overhead, ref.peak, ref.cache_mem)
        if table:
            m, a = sol.table()
            rm, ra = ref.table()
            np.testing.assert_array_equal(m, rm)
            np.testing.assert_array_equal(a, ra)
            table = False            # the table does not depend on the objective
    np.testing.assert_array_equal(fam.sets(), ref.sets())
    return fam


SMALL = ["chain16", "ladder40"]


@pytest.mark.parametrize("name", SMALL)
def test_small_cases(rc, oracle_mod, name):
    c = W.case(name)
    g = c.graph
    for B in (c.B, 2 * max(g.M), 2 * sum(g.M), 2 * sum(g.M) + 100):
        compare(rc, oracle_mod, g, c.mode, B)


def test_layered24_infeasible_and_feasible(rc, oracle_mod):
    c = W.case("layered24")
    g = c.graph
    compare(rc, oracle_mod, g, "exact", c.B)           # no strategy at B = 256
    for B in (900, 1200, 2 * sum(g.M)):
        compare(rc, oracle_mod, g, "exact", B)
        compare(rc, oracle_mod, g, "pruned", B)


RANDOM = [(n, p, seed) for seed, (n, p) in enumerate(
    [(n, p) for n in (2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12) for p in (0.1, 0.3, 0.5, 0.8)])]


@pytest.mark.parametrize("n,p,seed", RANDOM)
def test_random_dags(rc, oracle_mod, n, p, seed):
    g = W.random_dag(n, p, 1000 + seed, tmax=40, mmax=30)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for B in (lo - 1, lo, (2 * lo + hi) // 3, (lo + hi) // 2, hi):
        for mode in ("exact", "pruned"):
            compare(rc, oracle_mod, g, mode, B)


def test_wide_rows_many_tiles(rc, oracle_mod):
    """Rows far wider than one kernel tile, with ragged tails."""
    g = W.random_dag(9, 0.35, 77, tmax=900, mmax=40)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for B in (lo, (lo + hi) // 2, hi):
        compare(rc, oracle_mod, g, "exact", B)
        compare(rc, oracle_mod, g, "pruned", B)


def test_antichain_wide_levels(rc, oracle_mod):
    """Many independent targets per level (exact family of an antichain)."""
    g = W.antichain(9, seed=4, tmax=30, mmax=20)
    for B in (2 * max(g.M), sum(g.M), 2 * sum(g.M)):
        compare(rc, oracle_mod, g, "exact", B)


@pytest.mark.parametrize("path", ["level", "wavefront", "wide"])
def test_node_limit_antichain(rc, monkeypatch, path):
    """4096 nodes (64 words per set): the pruned family of an antichain, 4098
    sets (beyond the ghost-zone fill and the traceback's LDS arrays), whole
    table, t* and schedule against the closed form above, for both
    objectives, at the unconstrained budget, at one where only a two-segment
    chain fits, and at an infeasible one."""
    monkeypatch.setenv("RCDP_FILL", path)
    g = W.antichain(4096, seed=5, tmax=1, mmax=5)
    n, MV, TV = g.n, sum(g.M), sum(g.T)
    fam = rc.Graph.create(g).build_family("pruned")
    assert fam.info["num_sets"] == n + 2 and fam.info["num_pairs"] == 2 * n + 1
    big = max(g.M)
    for B in (2 * MV, 2 * (MV - big), 2 * (MV - big) - 1):
        em, ea, chain = antichain_pruned_expected(g, B)
        for objective in ("tc", "mc"):
            sol = fam.solve(B, objective)
            if chain is None:
                assert sol.status == rc.INFEASIBLE
            else:
                assert (sol.t_star, sol.m_star) == (TV, 0)
                for sched in reconstruct_each(sol, n + 2):
                    assert sched.chain.tolist() == chain
                    assert (sched.overhead, sched.cache_mem) == (TV, 0)
                    assert not sched.cached.any()
                    seg = np.full(n, len(chain) - 1)
                    if len(chain) == 2:
                        seg[chain[0] - 1] = 0
                        assert sched.peak == max(2 * big, 2 * (MV - big))
                    else:
                        assert sched.peak == 2 * MV
                    np.testing.assert_array_equal(sched.seg, seg)
            if objective == "tc":
                m, a = sol.table()
                np.testing.assert_array_equal(m, em, err_msg=f"B={B}")
                np.testing.assert_array_equal(a, ea, err_msg=f"B={B}")
            sol.free()


@pytest.mark.parametrize("path", ["level", "wide"])
def test_node_limit_chain(rc, monkeypatch, path):
    """A 4096-node chain with unit costs at an unconstrained budget: the
    pruned family is every prefix (4097 sets, 8.4 M pairs, 1.1e10
    relaxations).  A prefix's boundary is its last node, so caching every
    node but the sink takes all 4096 prefixes as the chain (the traceback at
    its longest) for the least overhead, 1 = T(sink) (reading 8's floor,
    cache memory n - 1, peak n + 1 in the last segment); overhead t needs
    n - t cached nodes, so row V is opt[V, t] = n - t for t >= 1; the
    memory-centric optimum is the one-segment chain (t = n, m = 0)."""
    monkeypatch.setenv("RCDP_FILL", path)
    n = 4096
    g = W.Graph(n, [[v + 1] if v + 1 < n else [] for v in range(n)], [1] * n, [1] * n)
    fam = rc.Graph.create(g).build_family("pruned")
    assert fam.info["num_sets"] == n + 1 and fam.info["num_pairs"] == n * (n + 1) // 2
    B = 2 * n
    sol = fam.solve(B, "tc")
    assert (sol.t_star, sol.m_star) == (1, n - 1)
    for sched in reconstruct_each(sol, n + 1):
        assert sched.chain.tolist() == list(range(1, n + 1))
        np.testing.assert_array_equal(sched.seg, np.arange(n))
        assert sched.cached.tolist() == [True] * (n - 1) + [False]
        assert (sched.overhead, sched.peak, sched.cache_mem) == (1, n + 1, n - 1)
    m, _ = sol.table(first=n, count=1)
    np.testing.assert_array_equal(m[0], np.array([-1] + [n - t for t in range(1, n + 1)]))
    sol.free()
    sol = fam.solve(B, "mc")
    assert (sol.t_star, sol.m_star) == (n, 0)
    for sched in reconstruct_each(sol, n + 1):
        assert sched.chain.tolist() == [n] and sched.overhead == n and sched.peak == 2 * n
    sol.free()


def test_empty_and_single(rc, oracle_mod):
    g0 = W.Graph(0, [], [], [])
    for mode in ("exact", "pruned"):
        gg = rc.Graph.create(g0)
        fam = gg.build_family(mode)
        assert fam.info["num_sets"] == 1
        sol = fam.solve(0, "tc")
        assert (sol.status, sol.t_star, sol.m_star) == (rc.OK, 0, 0)
        s = sol.reconstruct()
        assert len(s.chain) == 0 and (s.overhead, s.peak, s.cache_mem) == (0, 0, 0)
    g1 = W.chain(1, 3)
    for B in (2 * g1.M[0] - 1, 2 * g1.M[0], 10 ** 6):
        compare(rc, oracle_mod, g1, "exact", B)
        compare(rc, oracle_mod, g1, "pruned", B)


def test_budget_clamp_and_limits(rc, oracle_mod):
    g = W.chain(12, 5)
    gg = rc.Graph.create(g)
    fam = gg.build_family("exact")
    a = fam.solve(2 * sum(g.M), "tc").table()
    b = fam.solve(10 ** 9, "tc").table()               # clamped to 2 M(V)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    # memory sums the 32-bit cells cannot hold are refused when the graph is made
    with pytest.raises(rc.RcError) as e:
        rc.Graph.create(W.Graph(2, [[1], []], [3, 4], [1 << 28, 1 << 28]))
    assert e.value.status == rc.E_OVERFLOW
    with pytest.raises(rc.RcError) as e:
        rc.Graph.create(W.antichain(12)).build_family("exact", max_sets=4095)
    assert e.value.status == rc.E_TOO_MANY_SETS


# min(B, 2 M(V)) above 65532 does not fit the 16-bit cells: such a table
# takes 32-bit cells and the level fill.  Both sides of the boundary, and
# budgets far beyond it.
@pytest.mark.parametrize("B", [65532, 65533, 80000, 200000, 10 ** 6])
def test_budgets_beyond_16_bits(rc, oracle_mod, B):
    small = W.Graph(2, [[1], []], [3, 4], [20000, 20000])     # 2 M(V) = 80000
    big = W.Graph(2, [[1], []], [3, 4], [40000, 40000])       # 2 M(V) = 160000
    for g in (small, big):
        fam = compare(rc, oracle_mod, g, "exact", B)
        sol = fam.solve(B, "tc")
        wide = min(B, 2 * sum(g.M)) > 65532
        assert (sol.fill_kernel() == "k_fill_level") or not wide
        sol.free()


@pytest.mark.parametrize("n,p,seed", RANDOM[::3])
def test_random_dags_large_memory(rc, oracle_mod, n, p, seed):
    """Node memories in the tens of thousands: budgets on both sides of the
    16-bit boundary, both families, both objectives, whole tables."""
    g = W.random_dag(n, p, 4000 + seed, tmax=40, mmax=30000)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for B in sorted({lo, min(65532, hi), 65533, (lo + hi) // 2, hi}):
        if B < lo:
            continue
        for mode in ("exact", "pruned"):
            compare(rc, oracle_mod, g, mode, B)


def test_sweep_across_the_16_bit_boundary(rc, oracle_mod):
    """A batched sweep whose budgets straddle 65532: tables of both widths
    in one call, each as its own solve."""
    g = W.random_dag(9, 0.4, 4242, tmax=40, mmax=30000)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    assert lo < 65532 < hi
    budgets = [lo, 65532, 65533, hi]
    fam = rc.Graph.create(g).build_family("pruned")
    for B, sol in fam.sweep(budgets, "mc"):
        ref = oracle_mod.solve(g, "pruned", B, "mc")
        assert (sol.t_star, sol.m_star) == (ref.t_star, ref.m_star)
        m, _ = sol.table()
        np.testing.assert_array_equal(m, ref.table()[0])
        sol.free()


def test_dominance_beyond_16_bits(rc, oracle_mod):
    """The dominance skip's kernels keep 16-bit cells: a budget beyond them
    is refused with RC_E_OVERFLOW, one at the boundary is solved."""
    g = W.random_dag(8, 0.5, 4343, tmax=40, mmax=30000)
    B = 2 * sum(g.M)
    assert B > 65532
    fam = rc.Graph.create(g).build_family("exact")
    with pytest.raises(rc.RcError) as e:
        fam.solve_dominance(B)
    assert e.value.status == rc.E_OVERFLOW
    d = fam.solve_dominance(65532)
    ref = oracle_mod.solve(g, "exact", 65532, "tc")
    assert (d.t_star, d.m_star) == (ref.t_star, ref.m_star)


def test_largest_exact_family(rc, oracle_mod):
    """2^15 = 32768 lower sets (antichain of 15): the enumeration at scale."""
    g = W.antichain(15, seed=1, tmax=3, mmax=3)
    gg = rc.Graph.create(g)
    fam = gg.build_family("exact")
    assert fam.info["num_sets"] == 2 ** 15
    sets = fam.sets()
    vals = (sets * (1 << np.arange(15))).sum(axis=1)
    sizes = sets.sum(axis=1)
    order = np.lexsort((vals, sizes))
    np.testing.assert_array_equal(order, np.arange(2 ** 15))
    assert len(np.unique(vals)) == 2 ** 15


def test_repeatable(rc, oracle_mod):
    c = W.case("ladder40")
    gg = rc.Graph.create(c.graph)
    fam = gg.build_family("exact")
    first = fam.solve(c.B, "tc").table()
    for _ in range(3):
        again = fam.solve(c.B, "tc").table()
        np.testing.assert_array_equal(first[0], again[0])
        np.testing.assert_array_equal(first[1], again[1])


@pytest.mark.slow
@pytest.mark.parametrize("name", ["resnet50", "unet", "densenet121"])
def test_full_size_cases(rc, oracle_mod, name):
    """The CNN-shaped cases at full size, whole table."""
    c = W.case(name)
    compare(rc, oracle_mod, c.graph, c.mode, c.B, parallel=True)


# ---------------------------------------------------------------- fill paths
# The library picks a persistent wavefront fill for wide tables and
# per-level launches for narrow ones; RCDP_FILL forces one: "level", the
# row-push wavefront ("wavefront", fixed blocks of 8 targets), the
# split-panel wavefront ("wide", fixed blocks, panel records shared among
# waves) or the ghost-zone wavefront ("ghost", blocks cut to fit its
# recomputed halo).  Rows wider than one column make the wavefront's
# cross-workgroup waits real.

PATHS = ["level", "wavefront", "wide", "ghost"]

WIDE = [(n, p, seed) for seed, (n, p) in enumerate(
    [(n, p) for n in (4, 6, 8, 10, 12) for p in (0.2, 0.45, 0.7)])]


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("n,p,seed", WIDE)
def test_fill_paths_wide_rows(rc, oracle_mod, monkeypatch, path, n, p, seed):
    monkeypatch.setenv("RCDP_FILL", path)
    g = W.random_dag(n, p, 5000 + seed, tmax=700, mmax=60)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for B in (lo, (2 * lo + hi) // 3, hi):
        for mode in ("exact", "pruned"):
            compare(rc, oracle_mod, g, mode, B)


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("name", SMALL + ["layered24"])
def test_fill_paths_small_cases(rc, oracle_mod, monkeypatch, path, name):
    monkeypatch.setenv("RCDP_FILL", path)
    c = W.case(name)
    g = c.graph
    for B in (c.B, 2 * max(g.M), sum(g.M), 2 * sum(g.M)):
        compare(rc, oracle_mod, g, c.mode, B)


@pytest.mark.parametrize("path,kernel", [("level", "k_fill_level_vec"),
                                         ("wavefront", "k_fill_blocked"),
                                         ("wide", "k_fill_wide"), ("ghost", "k_fill_ghost")])
def test_fill_path_is_reported(rc, monkeypatch, path, kernel):
    """rc_solution_fill_path names the fill a forced RCDP_FILL ran."""
    monkeypatch.setenv("RCDP_FILL", path)
    g = W.random_dag(10, 0.45, 5007, tmax=700, mmax=60)
    fam = rc.Graph.create(g).build_family("exact")
    sol = fam.solve(2 * sum(g.M), "tc")
    assert sol.fill_kernel() == kernel
    sol.free()


@pytest.mark.parametrize("name,objective,kernel", [("densenet121", "tc", "k_trace_follow"),
                                                    ("resnet50_t10", "tc", "k_trace_follow"),
                                                    ("ladder40", "mc", "k_trace"),
                                                    ("unet", "mc", "k_trace")])
def test_trace_path_choice(rc, monkeypatch, name, objective, kernel):
    """The default traceback: the optarg slice where t* is small and the
    chain may be long, the predecessor scan where the slice's tests would
    cost more than the longest chain (the memory-centric optima, t* large);
    the schedule meets t*, opt[V, t*] and the budget either way."""
    monkeypatch.delenv("RCDP_TRACE", raising=False)
    c = W.case(name)
    fam = rc.Graph.create(c.graph).build_family(c.mode)
    sol = fam.solve(c.B, objective)
    assert sol.trace_kernel() is None
    sched = sol.reconstruct()
    assert sol.trace_kernel() == kernel
    assert (sched.overhead, sched.cache_mem) == (sol.t_star, sol.m_star) and sched.peak <= c.B
    sol.free()


def test_random_tracebacks(rc, oracle_mod):
    """Both tracebacks against the oracle's schedule on 300 seeded random
    DAGs (2-13 nodes, edge densities 0.1-0.85, small and large costs), a
    random budget around the feasible range, both families and objectives."""
    import random
    from tests.trace_paths import forced_trace, expected_kernel
    rng = random.Random(20261202)
    checked = 0
    for it in range(300):
        n = rng.randint(2, 13)
        p = rng.choice([0.1, 0.25, 0.4, 0.6, 0.85])
        g = W.random_dag(n, p, rng.randint(0, 10 ** 6), tmax=rng.choice([5, 40, 300]),
                         mmax=rng.choice([3, 30, 200]))
        lo, hi = 2 * max(g.M), 2 * sum(g.M)
        B = rng.randint(max(0, lo - 5), hi + 5)
        mode = rng.choice(["exact", "pruned"])
        fam = rc.Graph.create(g).build_family(mode)
        for objective in ("tc", "mc"):
            ref = oracle_mod.solve(g, mode, B, objective)
            sol = fam.solve(B, objective)
            assert (sol.t_star, sol.m_star) == (ref.t_star, ref.m_star), (it, B, mode, objective)
            if ref.status == oracle_mod.OK:
                chain, seg, cached = ref.schedule()
                for trace in ("scan", "slice"):
                    with forced_trace(trace):
                        sched = sol.reconstruct()
                    assert sol.trace_kernel() == expected_kernel(trace, ref.num_sets, sol.t_star)
                    np.testing.assert_array_equal(sched.chain, chain, err_msg=f"{it} {trace}")
                    np.testing.assert_array_equal(sched.seg, seg)
                    np.testing.assert_array_equal(sched.cached, cached)
                    assert (sched.overhead, sched.peak, sched.cache_mem) == (
                        ref.overhead, ref.peak, ref.cache_mem)
                    checked += 1
            sol.free()
        fam.free()
    assert checked > 400


@pytest.mark.parametrize("np_", ["1", "2", "4"])
@pytest.mark.parametrize("n,p,seed", WIDE[::2])
def test_wide_fill_panel_waves(rc, oracle_mod, monkeypatch, np_, n, p, seed):
    """The split-panel fill with one (the choice for launches of more
    columns than fit at once), two and four panel waves per workgroup."""
    monkeypatch.setenv("RCDP_FILL", "wide")
    monkeypatch.setenv("RCDP_WIDE_NP", np_)
    g = W.random_dag(n, p, 8000 + seed, tmax=900, mmax=60)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for B in (lo, (lo + hi) // 2, hi):
        for mode in ("exact", "pruned"):
            compare(rc, oracle_mod, g, mode, B)


@pytest.mark.parametrize("cpt", ["1", "2", "4"])
@pytest.mark.parametrize("n,p,seed", WIDE[::4])
def test_wavefront_column_widths(rc, oracle_mod, monkeypatch, cpt, n, p, seed):
    """The persistent fill at every column width (256, 512, 1024 cells)."""
    monkeypatch.setenv("RCDP_FILL", "wavefront")
    monkeypatch.setenv("RCDP_CPT", cpt)
    g = W.random_dag(n, p, 7000 + seed, tmax=900, mmax=60)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for B in (lo, (lo + hi) // 2, hi):
        for mode in ("exact", "pruned"):
            compare(rc, oracle_mod, g, mode, B)


@pytest.mark.parametrize("cpt", ["1", "2"])
@pytest.mark.parametrize("n,p,seed", WIDE[1::3])
def test_ghost_column_widths(rc, oracle_mod, monkeypatch, cpt, n, p, seed):
    """The ghost-zone fill at both column widths (256 and 576 owned cells
    plus the 64 recomputed ones), with rows of many columns."""
    monkeypatch.setenv("RCDP_FILL", "ghost")
    monkeypatch.setenv("RCDP_GHOST_CPT", cpt)
    g = W.random_dag(n, p, 7100 + seed, tmax=1500, mmax=60)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for B in (lo, (lo + hi) // 2, hi):
        for mode in ("exact", "pruned"):
            compare(rc, oracle_mod, g, mode, B)


@pytest.mark.parametrize("path", ["wavefront", "wide", "ghost"])
@pytest.mark.parametrize("seed", [10, 12, 16])
def test_wavefront_repeated_solves(rc, oracle_mod, monkeypatch, path, seed):
    """The same wide tables solved repeatedly: the persistent fill's columns
    meet in a different interleaving each time, and every table must match."""
    monkeypatch.setenv("RCDP_FILL", path)
    g = W.random_dag(12, 0.2, 5000 + seed, tmax=700, mmax=60)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for B in (lo, (2 * lo + hi) // 3, hi):
        for mode in ("exact", "pruned"):
            ref = oracle_mod.solve(g, mode, B, "tc")
            rm, _ = ref.table()
            fam = rc.Graph.create(g).build_family(mode)
            for rep in range(4):
                sol = fam.solve(B, "tc")
                m, _ = sol.table()
                np.testing.assert_array_equal(m, rm, err_msg=f"B={B} {mode} repetition {rep}")
                sol.free()


@pytest.mark.parametrize("path", ["wavefront", "wide", "ghost"])
@pytest.mark.parametrize("jitter", [1, 2, 3, 7])
def test_wavefront_race_delays(rc, oracle_mod, monkeypatch, path, jitter):
    """The race test: with RCDP_JITTER set, every wave of a persistent fill
    sleeps a pseudo-random time (drawn from the seed, its column, block and
    point) at one in four of its block starts and before a column publishes
    its progress, so that columns store, publish and poll in orders a plain
    run seldom takes.  Every table, t* and schedule must still be the
    oracle's, for both families at three budgets, and in a batch."""
    monkeypatch.setenv("RCDP_FILL", path)
    monkeypatch.setenv("RCDP_JITTER", str(jitter))
    g = W.random_dag(12, 0.45, 5100 + jitter, tmax=700, mmax=60)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for B in (lo, (2 * lo + hi) // 3, hi):
        for mode in ("exact", "pruned"):
            compare(rc, oracle_mod, g, mode, B)
    fam = rc.Graph.create(g).build_family("pruned")
    for B, sol in fam.sweep([lo, (lo + hi) // 2, hi], "tc"):
        rm, _ = oracle_mod.solve(g, "pruned", B, "tc").table()
        m, _ = sol.table()
        np.testing.assert_array_equal(m, rm, err_msg=f"batch B={B}")
        sol.free()


@pytest.mark.parametrize("path", PATHS)
def test_fill_paths_long_chain(rc, oracle_mod, monkeypatch, path):
    """A long chain: one target per level, rows of many columns."""
    monkeypatch.setenv("RCDP_FILL", path)
    g = W.chain(60, seed=9, tmax=400, mmax=30)
    for B in (2 * max(g.M), sum(g.M) // 3, sum(g.M), 2 * sum(g.M)):
        compare(rc, oracle_mod, g, "exact", B)


@pytest.mark.parametrize("n,p,seed", RANDOM[:16])
@pytest.mark.parametrize("mode", ["exact", "pruned"])
def test_min_budget_random(rc, oracle_mod, n, p, seed, mode):
    """rc_min_budget against the oracle's bisection (Section 5)."""
    g = W.random_dag(n, p, 1000 + seed, tmax=40, mmax=30)
    fam = rc.Graph.create(g).build_family(mode)
    assert fam.min_budget() == oracle_mod.min_budget(g, mode)


def test_min_budget_value_widths_and_large_families(rc, oracle_mod):
    """rc_min_budget where f needs 32 bits (2 M(V) above the 16-bit codes)
    and where the family's f table does not fit LDS (1024 sets)."""
    big = W.chain(6, seed=3, tmax=9, mmax=8)
    big = W.Graph(big.n, big.succ, big.T, [15000 + 997 * v for v in range(big.n)])
    assert 2 * sum(big.M) > 0xFFFF
    for mode in ("exact", "pruned"):
        fam = rc.Graph.create(big).build_family(mode)
        assert fam.min_budget() == oracle_mod.min_budget(big, mode)
    wide = W.antichain(10, seed=5, tmax=3, mmax=6)
    fam = rc.Graph.create(wide).build_family("exact")
    assert fam.info["num_sets"] == 1024
    assert fam.min_budget() == oracle_mod.min_budget(wide, "exact")


@pytest.mark.parametrize("name", ["chain16", "layered24", "ladder40", "unet", "resnet50",
                                  "densenet121"])
def test_min_budget_workloads(rc, name):
    """At every workload: the budget found is feasible and one less is not,
    both decided by the GPU solve; no budget below 2 max M_v can be feasible."""
    c = W.case(name)
    fam = rc.Graph.create(c.graph).build_family(c.mode)
    b = fam.min_budget()
    assert 2 * max(c.graph.M) <= b <= 2 * sum(c.graph.M)
    assert fam.solve(b, "tc").feasible
    assert not fam.solve(b - 1, "tc").feasible


@pytest.mark.slow
@pytest.mark.parametrize("name", ["layered24", "unet", "resnet50"])
def test_min_budget_oracle_full(rc, oracle_mod, name):
    c = W.case(name)
    fam = rc.Graph.create(c.graph).build_family(c.mode)
    assert fam.min_budget() == oracle_mod.min_budget(c.graph, c.mode)


def mc_budgets(b_min, m_total, count=32):
    """Budgets of the memory-centric sweep: count points from the smallest
    feasible budget to 2 M(V), where the one-segment chain is feasible."""
    top = 2 * m_total
    return [b_min + (j * (top - b_min)) // (count - 1) for j in range(count)]


@pytest.mark.slow
def test_mc_sweep_resnet50(rc, oracle_mod):
    """The memory-centric sweep of the ResNet-50-shaped graph over 32 budgets
    (Section 4.4) in one batched fill: at every budget t_MC, opt[V, t_MC],
    the traced chain, seg, cached and the Eq. 1 / Eq. 2 re-evaluation equal
    the oracle's; the whole table equals the oracle's at the smallest
    budget, two interior ones and 2 M(V); t_MC never decreases with the
    budget and reaches T(V) at 2 M(V)."""
    c = W.case("resnet50")
    g = c.graph
    fam = rc.Graph.create(g).build_family("pruned")
    b_min = fam.min_budget()
    assert b_min == oracle_mod.min_budget(g, "pruned", parallel=True)
    budgets = mc_budgets(b_min, sum(g.M))
    prev = -1
    for j, (B, sol) in enumerate(fam.sweep(budgets, "mc")):
        ref = oracle_mod.solve(g, "pruned", B, "mc", parallel=True)
        assert ref.status == oracle_mod.OK and sol.feasible, j
        assert (sol.t_star, sol.m_star) == (ref.t_star, ref.m_star), j
        sched = sol.reconstruct()
        chain, seg, cached = ref.schedule()
        np.testing.assert_array_equal(sched.chain, chain, err_msg=f"budget {j}")
        np.testing.assert_array_equal(sched.seg, seg)
        np.testing.assert_array_equal(sched.cached, cached)
        assert (sched.overhead, sched.peak, sched.cache_mem) == (
            ref.overhead, ref.peak, ref.cache_mem), j
        assert sched.peak <= B and sol.t_star >= prev
        prev = sol.t_star
        if j in (0, 10, 21, 31):
            m, a = sol.table()
            rm, ra = ref.table()
            np.testing.assert_array_equal(m, rm, err_msg=f"budget {j}")
            np.testing.assert_array_equal(a, ra, err_msg=f"budget {j}")
            del m, a, rm, ra
        del ref
        sol.free()
    assert prev == sum(g.T)


@pytest.mark.parametrize("name", ["resnet50_t10", "densenet121_t10", "unet_t10"])
def test_paper_cost_convention(rc, oracle_mod, name):
    """The CNN-shaped graphs with the forward times of the paper's experiments
    (T_v = 10 for convolutions, 1 otherwise): narrow tables, whole table and
    both objectives against the oracle, at the case budget and at the
    smallest feasible one."""
    c = W.case(name)
    compare(rc, oracle_mod, c.graph, c.mode, c.B)
    fam = rc.Graph.create(c.graph).build_family(c.mode)
    compare(rc, oracle_mod, c.graph, c.mode, fam.min_budget())


@pytest.mark.parametrize("path", PATHS + ["wide1"])
@pytest.mark.parametrize("n,p,seed", WIDE[2::5])
def test_solve_batch_tables(rc, oracle_mod, monkeypatch, path, n, p, seed):
    """rc_solve_batch: every budget's table, t* and schedule as the oracle's,
    the tables of all budgets filled in one pass ("wide1": the split-panel
    fill with one panel wave, the choice for large batched sweeps)."""
    monkeypatch.setenv("RCDP_FILL", "wide" if path == "wide1" else path)
    if path == "wide1":
        monkeypatch.setenv("RCDP_WIDE_NP", "1")
    g = W.random_dag(n, p, 5000 + seed, tmax=700, mmax=60)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    budgets = [lo, (3 * lo + hi) // 4, (lo + hi) // 2, hi, lo - 1]
    for mode in ("exact", "pruned"):
        fam = rc.Graph.create(g).build_family(mode)
        for objective in ("tc", "mc"):
            for B, sol in fam.sweep(budgets, objective):
                ref = oracle_mod.solve(g, mode, max(B, 0), objective)
                assert (sol.t_star, sol.m_star) == (ref.t_star, ref.m_star), (B, mode, objective)
                m, _ = sol.table()
                rm, _ = ref.table()
                np.testing.assert_array_equal(m, rm)
                if ref.status == oracle_mod.OK:
                    chain, _, _ = ref.schedule()
                    np.testing.assert_array_equal(sol.reconstruct().chain, chain)
                sol.free()
