"""Brute force over every chain of lower sets -- pins the oracle.

This is the naive exhaustive search of Section 4.1 of the paper, written
independently of the C oracle (Python, sets as int bitmasks, no DP table):
every increasing chain of family members starting at the empty set is
enumerated depth first, and each one is evaluated from the definitions of
Section 3 (the cache U_i is a union of boundaries, the overhead adds
T(V_i minus boundary(L_i)), the segment memory is Eq. 2).  A prefix is
extended only while every segment fits the budget, as the problem
statement requires.

From the enumeration it derives, per family member L and overhead t,
the least cache memory M(U) over all feasible chains ending at L with
overhead t (the definition of opt[L, t] in Section 4.2), and the smallest
family index of the penultimate set among the chains attaining it.
"""

from __future__ import annotations


def popcount(x):
    return bin(x).count("1")


def members(x):
    v = 0
    while x:
        if x & 1:
            yield v
        x >>= 1
        v += 1


class SetGraph:
    """A graph with bitmask neighbourhoods."""

    def __init__(self, g):
        self.g = g
        self.n = g.n
        self.full = (1 << g.n) - 1
        self.succ = [0] * g.n
        self.pred = [0] * g.n
        for v in range(g.n):
            for w in g.succ[v]:
                self.succ[v] |= 1 << w
                self.pred[w] |= 1 << v

    def cost(self, S, c):
        return sum(c[v] for v in members(S))

    def T(self, S):
        return self.cost(S, self.g.T)

    def M(self, S):
        return self.cost(S, self.g.M)

    def dplus(self, S):
        out = 0
        for v in members(S):
            out |= self.succ[v]
        return out

    def dminus(self, S):
        out = 0
        for v in members(S):
            out |= self.pred[v]
        return out

    def is_lower(self, L):
        return self.dminus(L) & ~L == 0

    def boundary(self, L):
        return self.dminus(self.full & ~L) & L

    def segment_memory(self, U_prev, L_prev, L):
        """Eq. 2 for segment V_i = L \\ L_prev with cache U_prev."""
        Vi = L & ~L_prev
        dp = self.dplus(L)
        return (self.M(U_prev) + 2 * self.M(Vi) + self.M(dp & ~L)
                + self.M(self.dminus(dp) & ~L))

    def sinks(self):
        return sum(1 << v for v in range(self.n) if self.succ[v] == 0)


def exact_family(sg):
    """All lower sets, by testing every subset (small n only)."""
    return sorted((S for S in range(1 << sg.n) if sg.is_lower(S)),
                  key=lambda S: (popcount(S), S))


def pruned_family(sg):
    """{L^v} plus the empty set and V; L^v = nodes from which v is reachable."""
    reach = [1 << v for v in range(sg.n)]       # reach[v] = ancestors of v and v
    changed = True
    while changed:
        changed = False
        for v in range(sg.n):
            new = reach[v]
            for p in members(sg.pred[v]):
                new |= reach[p]
            if new != reach[v]:
                reach[v] = new
                changed = True
    F = set(reach) | {0, sg.full}
    return sorted(F, key=lambda S: (popcount(S), S))


def family(sg, mode):
    return exact_family(sg) if mode == "exact" else pruned_family(sg)


def evaluate_chain(sg, chain_sets):
    """(overhead, peak, M(U_k)) of a chain of sets L_1..L_k (Eq. 1, Eq. 2)."""
    U = 0
    prev = 0
    peak = 0
    t = 0
    for L in chain_sets:
        peak = max(peak, sg.segment_memory(U, prev, L))
        bd = sg.boundary(L)
        t += sg.T((L & ~prev) & ~bd)
        U |= bd
        prev = L
    overhead = sg.T(sg.full & ~U)
    assert overhead == t        # Eq. 1: both sides of the identity
    return overhead, peak, sg.M(U)


def brute_table(g, mode, B, max_chains=5_000_000):
    """Enumerate every feasible chain prefix.

    Returns (F, opt, arg): F the family (bitmasks, family order); opt a dict
    (family index, t) -> least M(U); arg the matching dict of the smallest
    penultimate family index among prefixes attaining opt.
    """
    sg = SetGraph(g)
    F = family(sg, mode)
    index = {S: i for i, S in enumerate(F)}
    supers = [[j for j, S2 in enumerate(F) if S2 != S and S & ~S2 == 0] for S in F]
    opt = {(0, 0): 0}
    arg = {(0, 0): -1}
    count = 0
    # memo of per-set values used by every chain step (pure functions of sets)
    bd = [sg.boundary(S) for S in F]

    stack = [(0, 0, 0)]           # (family index of last set, t so far, U so far)
    while stack:
        i, t, U = stack.pop()
        L = F[i]
        for j in supers[i]:
            L2 = F[j]
            if sg.segment_memory(U, L, L2) > B:
                continue
            t2 = t + sg.T((L2 & ~L) & ~bd[j])
            U2 = U | bd[j]
            m2 = sg.M(U2)
            key = (j, t2)
            if key not in opt or m2 < opt[key] or (m2 == opt[key] and i < arg[key]):
                opt[key] = m2
                arg[key] = i
            count += 1
            if count > max_chains:
                raise RuntimeError("too many chains for brute force")
            stack.append((j, t2, U2))
    assert index[0] == 0
    return F, opt, arg


def select(opt, F, objective):
    """t* of the time-centric (min) or memory-centric (max) objective."""
    v = len(F) - 1
    ts = [t for (i, t) in opt if i == v]
    if not ts:
        return None
    return min(ts) if objective == "tc" else max(ts)


def brute_min_budget(g, mode, max_chains=5_000_000):
    """The smallest budget with a strategy: the least Eq. 2 peak over every
    chain of family sets from the empty set to V, by enumeration."""
    sg = SetGraph(g)
    F = family(sg, mode)
    supers = [[j for j, S2 in enumerate(F) if S2 != S and S & ~S2 == 0] for S in F]
    bd = [sg.boundary(S) for S in F]
    v = len(F) - 1
    best = None
    count = 0
    stack = [(0, 0, 0)]           # (family index of last set, U so far, peak so far)
    while stack:
        i, U, peak = stack.pop()
        if i == v:
            best = peak if best is None else min(best, peak)
            continue
        L = F[i]
        for j in supers[i]:
            p2 = max(peak, sg.segment_memory(U, L, F[j]))
            if best is not None and p2 >= best:
                continue
            count += 1
            if count > max_chains:
                raise RuntimeError("too many chains for brute force")
            stack.append((j, U | bd[j], p2))
    return 0 if v == 0 else best
