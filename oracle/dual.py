"""Memory-indexed form of Algorithm 1's recursion -- test infrastructure.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this module.  It shares nothing with the GPU library and nothing with the C
oracle: the family, the per-set and per-pair quantities are formed here from
their definitions in Sections 2-4 with numpy boolean arrays over node ids.

Algorithm 1 (Section 4.2, Appendix A) walks states (L, t, m): a chain that
ends at lower set L with forward time t and cached memory m = M(U).  A
transition L -> L' (L a proper subset of L') is allowed when m + c <= B,
c = 2 M(L' \\ L) + M(delta+(L') \\ L') + M(delta-(delta+(L')) \\ L') (Eq. 2),
and leads to (L', t + T((L' \\ L) \\ boundary(L')), m + M(boundary(L') \\ L)).
Algorithm 1 keeps, per (L, t), the least m; the budget test is monotone in
m, so nothing reachable in t is lost.  The same reachable set can be kept per
(L, m) instead: the least t for the time-centric objective (a later step adds
the same time to either state, so the faster one is never worse), the
greatest t for the memory-centric one (Section 4.4).  Then

    t*  = min over m of  tmin[V, m],   t_MC = max over m of tmax[V, m],

and opt[V, t*] of Algorithm 1 is the least m with tmin[V, m] = t* (resp.
tmax[V, m] = t_MC).  Rows run over m in [0, min(B, M(V))]: every cached
memory is a sum of distinct node memories (m = M(U), U a subset of V).

A chain attaining the optimum is traced back through the table (Section
4.2's traceback read on cells (L, m)) and re-evaluated from the definitions
of Section 3 (evaluate_chain).

Pinned by tests/test_oracle_dual.py: t* and opt[V, t*] against Algorithm 1
(the C oracle) and against brute force over every chain
(tests/bruteforce.py); the traced chain by its re-evaluation (overhead = t*,
M(U_k) = opt[V, t*], every segment within B) and by the C oracle's
evaluation of the same chain; the family order against the C oracle's; and
planted mistakes in the table and in the evaluation.
"""

import numpy as np

INF = np.iinfo(np.int64).max // 4


def _adjacency(g):
    n = g.n
    succ = np.zeros((n, n), dtype=bool)
    for v in range(n):
        for w in g.succ[v]:
            succ[v, w] = True
    return succ


def _topo(succ):
    """Kahn's order of the DAG."""
    n = succ.shape[0]
    indeg = succ.sum(axis=0).astype(int)
    order = [v for v in range(n) if indeg[v] == 0]
    k = 0
    while k < len(order):
        v = order[k]
        k += 1
        for w in np.flatnonzero(succ[v]):
            indeg[w] -= 1
            if indeg[w] == 0:
                order.append(int(w))
    if len(order) != n:
        raise ValueError("the graph has a cycle")
    return order


def _ancestors(succ, order):
    """anc[v]: v and every node with a path to v (Section 4.3's L^v)."""
    n = succ.shape[0]
    anc = np.eye(n, dtype=bool)
    for v in order:                      # predecessors first
        for p in np.flatnonzero(succ[:, v]):
            anc[v] |= anc[p]
    return anc


def _lower_sets(succ, order):
    """Every set closed under predecessors, by deciding the nodes in
    topological order (a node may join only after all its predecessors)."""
    n = succ.shape[0]
    preds = [np.flatnonzero(succ[:, v]) for v in range(n)]
    out = []
    cur = np.zeros(n, dtype=bool)

    def rec(k):
        if k == n:
            out.append(cur.copy())
            return
        v = order[k]
        rec(k + 1)                       # v left out
        if all(cur[p] for p in preds[v]):
            cur[v] = True
            rec(k + 1)
            cur[v] = False

    rec(0)
    return out


def family(g, mode):
    """The family as a bool array [F, n] in the canonical order: ascending
    size, equal sizes by ascending numeric value sum of 2^v over the set
    (the order Algorithm 1's loop takes; the optimum does not depend on it,
    the traced chain's tie rule does).  mode "pruned": the ancestor closures
    plus the empty set and V (Section 4.3); "exact": every lower set
    (Section 4.2), by enumeration, for small graphs only."""
    n = g.n
    succ = _adjacency(g)
    order = _topo(succ)
    if mode == "pruned":
        sets = [np.zeros(n, bool)] + list(_ancestors(succ, order)) + [np.ones(n, bool)]
    elif mode == "exact":
        if n > 40:
            raise ValueError("exact family enumeration is for small graphs")
        sets = _lower_sets(succ, order)
    else:
        raise ValueError(mode)
    seen, out = set(), []
    for L in sets:
        key = L.tobytes()
        if key not in seen:
            seen.add(key)
            out.append(L)
    out.sort(key=lambda L: (int(L.sum()), sum(1 << int(v) for v in np.flatnonzero(L))))
    return np.array(out, dtype=bool).reshape(len(out), n), succ


def evaluate_chain(g, S, chain):
    r"""Eq. 1 and Eq. 2 of the canonical strategy of the chain L_1 < ... < L_k
    (family indices into S), from their definitions (Section 3): V_i =
    L_i \ L_{i-1}, U_i = U_{i-1} + boundary(L_i); segment i needs
    M(U_{i-1}) + 2 M(V_i) + M(delta+(L_i) \ L_i) + M(delta-(delta+(L_i)) \ L_i);
    the overhead is T(V \ U_k).  Returns (seg, cached, overhead, peak, M(U_k))."""
    n = g.n
    succ = _adjacency(g)
    pred = succ.T
    T = np.asarray(g.T, dtype=np.int64)
    M = np.asarray(g.M, dtype=np.int64)
    seg = np.full(n, -1, dtype=np.int32)
    U = np.zeros(n, dtype=bool)
    prev = np.zeros(n, dtype=bool)
    peak = 0
    for i, idx in enumerate(chain):
        L = S[idx]
        Vi = L & ~prev
        seg[Vi] = i
        dp = succ[L].any(axis=0) if L.any() else np.zeros(n, bool)
        dmdp = pred[dp].any(axis=0) if dp.any() else np.zeros(n, bool)
        mem = M[U].sum() + 2 * M[Vi].sum() + M[dp & ~L].sum() + M[dmdp & ~L].sum()
        peak = max(peak, int(mem))
        U |= L & succ[:, ~L].any(axis=1)
        prev = L
    return seg, U.copy(), int(T[~U].sum()), peak, int(M[U].sum())


def solve(g, mode, B, objective="tc"):
    """(t, m) of the objective, or None when no chain reaches V within B,
    and a chain that attains it.

    Returns a dict with t, m, the family size, the number of pairs, the
    relaxations done (one per (pair, m) with m inside the budget window) and,
    when feasible, the chain traced back through the table (from (V, m, t):
    the smallest family index L whose cell (L, m - dm) passes the budget test
    and holds t - dt; along an optimal chain one always does) with its seg,
    cached, overhead, peak and M(U_k) re-evaluated by evaluate_chain."""
    if B < 0:
        raise ValueError("B < 0")
    S, succ = family(g, mode)
    F, n = S.shape
    T = np.asarray(g.T, dtype=np.int64)
    M = np.asarray(g.M, dtype=np.int64)
    width = int(min(B, M.sum())) + 1
    pred = succ.T

    bd = np.array([L & (succ[:, ~L].any(axis=1)) for L in S])          # boundary(L)
    out = np.zeros(F, dtype=np.int64)
    for j in range(F):
        L = S[j]
        dp = succ[L].any(axis=0)                                       # delta+(L)
        dmdp = pred[dp].any(axis=0) if dp.any() else np.zeros(n, bool)  # delta-(delta+(L))
        out[j] = M[dp & ~L].sum() + M[dmdp & ~L].sum()

    tc = objective == "tc"
    unreached = INF if tc else -1
    D = np.full((F, width), unreached, dtype=np.int64)
    D[0, 0] = 0                                                       # (empty set, t = 0, m = 0)
    def pair(i, j):
        """c, dt, dm of the pair L < L' (None unless L is a proper subset)."""
        L, Lp = S[i], S[j]
        if not (Lp & ~L).any() or (L & ~Lp).any():
            return None
        Vp = Lp & ~L
        return (int(2 * M[Vp].sum() + out[j]), int(T[Vp & ~bd[j]].sum()),
                int(M[bd[j] & ~L].sum()))

    pairs = 0
    relax = 0
    for i in range(F):                   # sources in ascending size: every proper subset first
        for j in range(F):
            q = pair(i, j)
            if q is None:
                continue
            pairs += 1
            c, dT, dM = q
            # source m with m + c <= B; also m + dM <= M(V), which every
            # reachable m meets (m = M(U) with U inside L, disjoint from the
            # added boundary), so the clip drops no reachable state
            top = min(B - c, width - 1 - dM)
            if top < 0:
                continue
            src = D[i, :top + 1]
            dst = D[j, dM:dM + top + 1]
            relax += top + 1
            if tc:
                cand = np.where(src < INF, src + dT, INF)
                np.minimum(dst, cand, out=dst)
            else:
                cand = np.where(src >= 0, src + dT, -1)
                np.maximum(dst, cand, out=dst)
    row = D[F - 1]
    reach = row < INF if tc else row >= 0
    result = {"sets": F, "pairs": pairs, "relaxations": relax, "width": width}
    if not reach.any():
        result.update(t=None, m=None)
        return result
    t = int(row[reach].min()) if tc else int(row[reach].max())
    m = int(np.flatnonzero(row == t)[0])
    result.update(t=t, m=m)
    chain = []
    j, mj, tj = F - 1, m, t
    while j != 0:
        step = None
        for i in range(F):
            q = pair(i, j)
            if q is None:
                continue
            c, dT, dM = q
            ms = mj - dM
            if ms < 0 or ms > B - c or ms >= width:
                continue
            v = int(D[i, ms])
            if (v < INF if tc else v >= 0) and v + dT == tj:
                step = (i, ms, v)
                break
        assert step is not None, "no predecessor reproduces the cell"
        chain.append(j)
        j, mj, tj = step
    assert (mj, tj) == (0, 0), "the chain must start at (empty set, 0, 0)"
    chain = chain[::-1]
    seg, cached, overhead, peak, cache_mem = evaluate_chain(g, S, chain)
    result.update(chain=chain, seg=seg, cached=cached, overhead=overhead, peak=peak,
                  cache_mem=cache_mem)
    return result
