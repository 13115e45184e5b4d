"""Pin the oracle's dominance skip (Section 4.2, last paragraph).

The skip: an entry opt[L, t'] is not propagated when some t < t' of the same
row has opt[L, t] < opt[L, t'].  Read for the time-centric objective only
(the memory-centric one wants the largest reachable t, which a skipped entry
may be the only way to reach).

What the mathematics fixes, and is checked here:

* Each row's weak front, the entries (t, m) with m <= opt[L, u] for every
  u < t, is the same with and without the skip.  (A front entry of L' comes
  from a front entry of its source row: a source with an earlier, strictly
  smaller entry would give L' an earlier, strictly smaller one.)  Hence t*
  and opt[V, t*] are unchanged, and every entry of the skipped table is at
  least the full table's.
* Exactly: skipped[L', t'] is the least m + dM over pairs L < L' and front
  entries (t, m) of row L (taken from brute force over every chain,
  tests/bruteforce.py) with m + c <= B and t + dT = t'.  The skipped table
  must equal this cell for cell, finite set included.
* The chain traced back through the skipped table re-evaluates (Eq. 1, Eq.
  2) to overhead t*, cache M(U_k) = opt[V, t*] and every segment within B.

Planted mistakes in a copy of the C oracle (an inverted comparison, a
running minimum never updated or replaced by the previous entry alone,
a non-strict skip) each
fail the exact pin.
"""

import subprocess

import numpy as np
import pytest

from oracle import oracle as O
from paper_1905_11722_amd import workloads as W
from tests import bruteforce as bf

SRC = O.__file__.replace("oracle.py", "rc_oracle.c")


def _finite(r):
    opt, _ = r.table()
    return {(int(i), int(t)): int(opt[i, t]) for i, t in zip(*np.nonzero(opt >= 0))}


def _front(entries):
    """Weak front of one row given as {t: m}: m <= every earlier m."""
    out, least = [], None
    for t in sorted(entries):
        m = entries[t]
        if least is None or m <= least:
            out.append((t, m))
        least = m if least is None else min(least, m)
    return out


def _rows(table):
    rows = {}
    for (i, t), m in table.items():
        rows.setdefault(i, {})[t] = m
    return rows


def closed_form(g, mode, B):
    """The skipped table from brute force's full table, one step per pair."""
    sg = bf.SetGraph(g)
    F, bopt, _ = bf.brute_table(g, mode, B)
    rows = _rows(bopt)
    want = {(0, 0): 0}
    for j, Lp in enumerate(F):
        if j == 0:
            continue
        bd = sg.boundary(Lp)
        dp = sg.dplus(Lp)
        out = sg.M(dp & ~Lp) + sg.M(sg.dminus(dp) & ~Lp)
        for i, L in enumerate(F):
            if L == Lp or L & ~Lp:
                continue
            Vp = Lp & ~L
            c = 2 * sg.M(Vp) + out
            dT = sg.T(Vp & ~bd)
            dM = sg.M(bd & ~L)
            for t, m in _front(rows.get(i, {})):
                if m + c > B:
                    continue
                key = (j, t + dT)
                if key not in want or m + dM < want[key]:
                    want[key] = m + dM
    return F, bopt, want


TINY = [W.random_dag(n, p, s, tmax=9, mmax=7)
        for n, p, s in [(5, 0.3, 1), (6, 0.5, 2), (6, 0.2, 3), (7, 0.4, 4), (4, 0.6, 5), (7, 0.25, 6)]]
TINY += [W.ladder(3, seed=2, tmax=9, mmax=9), W.layered(3, 2, seed=1, tmax=9, mmax=9)]
# memories of 1 or 2: tied entries of one row that are the only source of
# some cell (strict vs non-strict comparison), and rows whose memory is not
# monotone past the running minimum (running minimum vs previous entry)
TINY += [W.random_dag(n, p, s, tmax=9, mmax=2) for n, p, s in [(7, 0.35, 0), (7, 0.35, 1), (7, 0.35, 2), (6, 0.5, 2)]]


def _budgets(g):
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    return (lo, (2 * lo + hi) // 3, (lo + hi) // 2, hi)


def exact_pins_hold(lib=None):
    """The exact closed form and t*, m* on the tiny graphs; False on the first
    failure.  lib: a mutant library to run instead of the oracle's."""
    with O.using(lib if lib is not None else O._load()):
        for g in TINY:
            for B in _budgets(g):
                for mode in ("exact", "pruned"):
                    F, bopt, want = closed_form(g, mode, B)
                    r = O.solve_dominance(g, mode, B)
                    if r.status not in (O.OK, O.INFEASIBLE):
                        return False
                    if _finite(r) != want:
                        return False
                    ts = bf.select(bopt, F, "tc")
                    if ts is None:
                        if r.status != O.INFEASIBLE:
                            return False
                        continue
                    if (r.t_star, r.m_star) != (ts, bopt[(len(F) - 1, ts)]):
                        return False
        return True


def test_exact_closed_form_on_tiny_graphs():
    assert exact_pins_hold()


def _compare(g, mode, B):
    full = O.solve(g, mode, B, "tc")
    skip = O.solve_dominance(g, mode, B)
    assert skip.status == full.status
    assert (skip.t_star, skip.m_star) == (full.t_star, full.m_star)
    a, b = _finite(full), _finite(skip)
    assert set(b) <= set(a)
    assert all(b[k] >= a[k] for k in b)
    ra, rb = _rows(a), _rows(b)
    for i in ra:
        assert _front(ra[i]) == _front(rb.get(i, {})), i
    if skip.status == O.OK:
        chain, _, _ = skip.schedule()
        assert skip.evaluate_chain(chain) == (skip.overhead, skip.peak, skip.cache_mem)
        assert (skip.overhead, skip.cache_mem) == (skip.t_star, skip.m_star) and skip.peak <= B
    return len(a), len(b)


@pytest.mark.parametrize("seed", range(10))
def test_random_dags_keep_fronts_and_optimum(seed):
    g = W.random_dag(10, 0.3, 500 + seed, tmax=30, mmax=20)
    lo, hi = 2 * max(g.M), 2 * sum(g.M)
    for mode in ("exact", "pruned"):
        for B in (0, lo - 1, lo, (lo + hi) // 2, hi, 10 ** 6):
            _compare(g, mode, B)


@pytest.mark.parametrize("name", ["chain16", "layered24", "ladder40", "unet_t10"])
def test_workloads_keep_fronts_and_optimum(name):
    c = W.case(name)
    n_full, n_skip = _compare(c.graph, c.mode, c.B)
    assert n_skip <= n_full


def test_the_skip_removes_entries():
    """On the 40-rung ladder the skip leaves markedly fewer finite entries."""
    c = W.case("ladder40")
    n_full, n_skip = _compare(c.graph, c.mode, c.B)
    assert n_skip < 0.8 * n_full


def test_arguments():
    g = W.chain(4, 1)
    assert O.solve_dominance(g, 2, 100).status == O.E_ARG          # no such family
    assert O.solve_dominance(g, "exact", -1).status == O.E_ARG
    assert O.solve_dominance(W.Graph(0, [], [], []), "exact", 0).t_star == 0


MUTANTS = {
    "inverted": ("dominance_skip && least < m;", "dominance_skip && least > m;"),
    "never_updated": ("if (m < least) least = m;", "(void)least;"),
    "previous_only": ("if (m < least) least = m;", "least = m;"),
    "non_strict": ("dominance_skip && least < m;", "dominance_skip && least <= m;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, name
    mutated = tmp_path / "mutant.c"
    mutated.write_text(src.replace(old, new))
    lib_path = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O1", "-std=c99", "-shared", "-fPIC", str(mutated), "-o", str(lib_path)])
    assert not exact_pins_hold(O.open_library(str(lib_path))), name
