"""The pins are sharp: each planted mistake in a copy of the oracle fails them.

Every mutant below is a plausible slip in transcribing Algorithm 1 or the
definitions of Sections 2-4 (a dropped term of Eq. 2, a wrong comparison,
a wrong set in a difference, a reversed order ...).  The mutant source is
compiled to a temporary library and run through a quick subset of the pins
(brute force over chains, the chain closed form, the objective ceilings).
All mistakes are planted on the CPU, in the oracle only.
"""

import os
import subprocess

import numpy as np
import pytest

from oracle import oracle as O
from paper_1905_11722_amd import workloads as W
from tests import bruteforce as bf

SRC = os.path.join(os.path.dirname(O.__file__), "rc_oracle.c")

MUTANTS = {
    "drop_term_iv": ("outm[j] = cost_sum(n, dpo, g.M) + cost_sum(n, dmo, g.M);",
                     "outm[j] = cost_sum(n, dpo, g.M);"),
    "drop_term_iii": ("outm[j] = cost_sum(n, dpo, g.M) + cost_sum(n, dmo, g.M);",
                      "outm[j] = cost_sum(n, dmo, g.M);"),
    "single_segment_memory": ("2 * cost_sum(n, Vp, g.M) + outm[j]", "cost_sum(n, Vp, g.M) + outm[j]"),
    "budget_ge": ("if (Mcal > B) continue;", "if (Mcal >= B) continue;"),
    "nonstrict_update": ("if (optLp[tp] > mp) {", "if (optLp[tp] >= mp) {"),
    "dM_minus_Lprime": ("set_minus(n, bd, L, bdl);", "set_minus(n, bd, Lp, bdl);"),
    "dT_keeps_boundary": ("set_minus(n, Vp, bd, Vpb);", "set_minus(n, Vp, L, Vpb);"),
    "boundary_uses_dplus": ("  delta_minus(g, comp, dm);\n  set_and", "  delta_plus(g, comp, dm);\n  set_and"),
    "order_reversed": ("if (A[v] != B[v]) return A[v] < B[v] ? -1 : 1;",
                       "if (A[v] != B[v]) return A[v] < B[v] ? 1 : -1;"),
    "mc_takes_min": ("if (ts < 0 || objective == 1) ts = t;", "if (ts < 0) ts = t;"),
    "pruned_without_V": ("if (!have && n > 0) family_push(&f, tmp);", "(void)have;"),
    "eq2_drops_cache": ("int64_t mem = cost_sum(n, U, g->M) + 2 * cost_sum(n, Vi, g->M) +",
                        "int64_t mem = 2 * cost_sum(n, Vi, g->M) +"),
    "descendant_sets": ("if (g->adj[p * n + x] && !out[p]) { out[p] = 1; stack[top++] = p; }",
                        "if (g->adj[x * n + p] && !out[p]) { out[p] = 1; stack[top++] = p; }"),
}


def quick_pins_hold(lib):
    """A fast subset of the pins; False as soon as one fails."""
    with O.using(lib):
        graphs = [W.random_dag(n, p, s, tmax=9, mmax=7)
                  for n, p, s in [(5, 0.3, 1), (6, 0.5, 2), (6, 0.2, 3), (7, 0.4, 4), (4, 0.6, 5)]]
        graphs.append(W.ladder(3, seed=2, tmax=9, mmax=9))
        graphs.append(W.layered(3, 2, seed=1, tmax=9, mmax=9))
        for g in graphs:
            lo, hi = 2 * max(g.M), 2 * sum(g.M)
            for B in (lo, (2 * lo + hi) // 3, (lo + hi) // 2, hi):
                for mode in ("exact", "pruned"):
                    F, bopt, barg = bf.brute_table(g, mode, B)
                    r = O.solve(g, mode, B, "tc")
                    fam = [sum(1 << v for v in range(g.n) if row[v]) for row in r.sets()]
                    if fam != F:
                        return False
                    opt, arg = r.table()
                    for (i, t), m in bopt.items():
                        if opt[i, t] != m or arg[i, t] != barg[(i, t)]:
                            return False
                    if int((opt >= 0).sum()) != len(bopt):
                        return False
                    for obj in ("tc", "mc"):
                        ts = bf.select(bopt, F, obj)
                        ro = O.solve(g, mode, B, obj)
                        if ts is None:
                            if ro.status != O.INFEASIBLE:
                                return False
                            continue
                        if ro.t_star != ts:
                            return False
                        chain, _, _ = ro.schedule()
                        got = bf.evaluate_chain(bf.SetGraph(g), [F[c] for c in chain])
                        if got != (ro.overhead, ro.peak, ro.cache_mem):
                            return False
            # Eq. 1 / Eq. 2 of arbitrary chains through the family
            r = O.solve(g, "exact", hi, "tc")
            F = [sum(1 << v for v in range(g.n) if row[v]) for row in r.sets()]
            rng = np.random.default_rng(g.n)
            for _ in range(10):
                chain, cur = [], 0
                while cur != F[-1]:
                    ups = [j for j, S in enumerate(F) if S != cur and cur & ~S == 0]
                    j = int(rng.choice(ups))
                    chain.append(j)
                    cur = F[j]
                if r.evaluate_chain(chain) != bf.evaluate_chain(bf.SetGraph(g), [F[c] for c in chain]):
                    return False
        return True



def test_unmutated_oracle_passes():
    assert quick_pins_hold(O._load())


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site of {name} not unique"
    mutated = tmp_path / "mutant.c"
    mutated.write_text(src.replace(old, new))
    lib_path = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O1", "-std=c99", "-shared", "-fPIC", str(mutated), "-o", str(lib_path)])
    lib = O.open_library(str(lib_path))
    assert not quick_pins_hold(lib), f"mutant {name} slipped through the pins"
