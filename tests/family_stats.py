"""The DP's unit of work and table size, counted from the oracle's family
with plain set operations -- test infrastructure.

A relaxation is one (L, L', t) of Algorithm 1 (Appendix A) with L a proper
subset of L' (both in the family) and t inside the range where opt[L, t] can
be finite, 0 <= t <= T(L \\ boundary(L)): every node a chain ending at L
recomputes lies in L \\ boundary(L) (Eq. 1 charges V_i \\ boundary(L_i) per
segment), so larger t are never reached.  So

    w_L          = T(L \\ boundary(L)) + 1          (cells of row L)
    table_cells  = sum over the family of w_L
    relaxations  = sum over pairs (L, L') of w_L

with boundary(L) = {v in L : some successor of v is outside L} (Section 2).
"""

import numpy as np

from oracle import oracle as O


def stats_from_sets(graph, sets):
    """Counts of the family given as a bool array [F, n] in family order."""
    n = graph.n
    F = len(sets)
    T = np.asarray(graph.T, dtype=np.int64)
    succ = np.zeros((n, n), dtype=bool)
    for v in range(n):
        for w in graph.succ[v]:
            succ[v, w] = True
    w = np.empty(F, dtype=np.int64)
    for s in range(F):
        L = sets[s]
        outside = succ[:, ~L].any(axis=1) if n else np.zeros(0, bool)
        bd = L & outside
        w[s] = T[L & ~bd].sum() + 1
    # L_i proper subset of L_j: no node of L_i outside L_j, and L_i != L_j
    S = sets.astype(np.int32)
    inside = (S @ (1 - S).T) == 0 if n else np.ones((F, F), bool)
    np.fill_diagonal(inside, False)
    pairs_i = inside.sum(axis=1)            # supersets of each source
    return {
        "num_sets": int(F),
        "num_pairs": int(inside.sum()),
        "table_cells": int(w.sum()),
        "relaxations": int((pairs_i * w).sum()),
        "max_row": int(w.max()) if F else 0,
        "T_total": int(T.sum()),
        "w": w,
    }


def family_stats(graph, mode):
    fam = O.family(graph, mode)
    assert fam.status == O.OK, fam.status
    return stats_from_sets(graph, fam.sets())
