"""Closed forms of the DP on graphs simple enough to solve by hand -- test
infrastructure.  They share nothing with the oracle or the HIP path; a CPU
test pins each against the oracle on small inputs, and the GPU tests use them
where the oracle would take minutes (the node limit)."""

import numpy as np


def antichain_pruned_expected(g, B):
    """Closed form of the pruned family of an antichain (no edges) of n >= 2
    nodes (with one node, V is the one ancestor set), for a
    check at the node limit where the oracle's subset tests over 4096-node
    sets take minutes.  The family is the empty set, the singletons {v}
    (family index 1 + v: equal sizes in ascending numeric value) and V.  No
    node has a successor, so every boundary is empty and nothing is ever
    cached (every finite cell holds 0); a chain's overhead is T(V) whatever
    its cuts (Eq. 1), row {v} is finite only at t = T_v (from the empty set,
    if 2 M_v <= B) and row V only at T(V): by the one-segment chain (peak
    2 M(V)) or by empty -> {v} -> V (peaks 2 M_v and 2 (M(V) - M_v), Eq. 2
    with A = 0).  optarg is the smallest predecessor index (reading 2).
    Returns (m, arg) over t = 0..T(V) (-1 = infinite / none) and the chain."""
    n, T, M = g.n, g.T, g.M
    TV, MV = sum(T), sum(M)
    F = n + 2
    m = np.full((F, TV + 1), -1, dtype=np.int64)
    a = np.full((F, TV + 1), -1, dtype=np.int32)
    m[0, 0] = 0
    for v in range(n):
        if 2 * M[v] <= B:
            m[1 + v, T[v]], a[1 + v, T[v]] = 0, 0
    chain = None
    if 2 * MV <= B:
        m[F - 1, TV], a[F - 1, TV] = 0, 0
        chain = [F - 1]
    else:
        for v in range(n):
            if 2 * M[v] <= B and 2 * (MV - M[v]) <= B:
                m[F - 1, TV], a[F - 1, TV] = 0, 1 + v
                chain = [1 + v, F - 1]
                break
    return m, a, chain
