"""ctypes wrapper of the C oracle (``rc_oracle.c``) -- test infrastructure.

``solve(graph, mode, B, objective)`` runs Algorithm 1 of the paper
(Appendix A) on the CPU and returns an :class:`OracleResult` holding the
family, the whole opt / optarg table (rows on demand), t*, m* = opt[V, t*],
the traced chain and its re-evaluated Eq. 1 overhead and Eq. 2 peak.
"""

import contextlib
import ctypes
import os

import numpy as np

from . import build as _build

OK, INFEASIBLE = 0, 1
E_ARG, E_CYCLE, E_COST, E_TOO_MANY_SETS, E_OVERFLOW, E_NOMEM, E_INTERNAL = -1, -2, -3, -4, -5, -6, -8
MODES = {"exact": 0, "pruned": 1}
OBJECTIVES = {"tc": 0, "mc": 1}

_libs = {}


def _load(parallel=False):
    """The single-threaded library, or (parallel=True) the OpenMP build of
    the same source, whose results are identical."""
    if parallel in _libs:
        return _libs[parallel]
    path = _build.LIB_OMP if parallel else _build.LIB
    if not os.path.exists(path):
        _build.build()
    _libs[parallel] = open_library(path)
    return _libs[parallel]


@contextlib.contextmanager
def using(lib):
    """Run the single-threaded entry points on another compiled copy of the
    oracle (a planted-mistake build in the tests) inside the block."""
    saved = _libs.get(False)
    _libs[False] = lib
    try:
        yield
    finally:
        if saved is None:
            _libs.pop(False, None)
        else:
            _libs[False] = saved


def threads(parallel=True):
    """Threads the oracle's fill runs on in that build."""
    return _load(parallel).oracle_threads()


def open_library(path):
    """Load a compiled oracle library and declare its C signatures."""
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i32p = ctypes.POINTER(ctypes.c_int32)
    i64p = ctypes.POINTER(ctypes.c_int64)
    lib.oracle_solve.restype = P
    lib.oracle_solve.argtypes = [ctypes.c_int, i32p, i32p, i64p, i64p, ctypes.c_int,
                                 ctypes.c_int64, ctypes.c_int, ctypes.c_int64, ctypes.c_int64]
    lib.oracle_family.restype = P
    lib.oracle_family.argtypes = [ctypes.c_int, i32p, i32p, i64p, i64p, ctypes.c_int,
                                  ctypes.c_int64]
    lib.oracle_solve_dominance.restype = P
    lib.oracle_solve_dominance.argtypes = [ctypes.c_int, i32p, i32p, i64p, i64p, ctypes.c_int,
                                           ctypes.c_int64, ctypes.c_int64]
    for name, rt in [("oracle_status", ctypes.c_int), ("oracle_num_sets", ctypes.c_int64),
                     ("oracle_T_total", ctypes.c_int64), ("oracle_num_pairs", ctypes.c_int64),
                     ("oracle_relaxations_literal", ctypes.c_int64),
                     ("oracle_t_star", ctypes.c_int64), ("oracle_m_star", ctypes.c_int64),
                     ("oracle_k", ctypes.c_int32), ("oracle_overhead", ctypes.c_int64),
                     ("oracle_peak", ctypes.c_int64), ("oracle_cache_mem", ctypes.c_int64)]:
        f = getattr(lib, name)
        f.restype = rt
        f.argtypes = [P]
    lib.oracle_get_sets.argtypes = [P, P]
    lib.oracle_get_rows.argtypes = [P, ctypes.c_int64, ctypes.c_int64, P, P]
    lib.oracle_get_schedule.argtypes = [P, P, P, P]
    lib.oracle_evaluate_chain.restype = ctypes.c_int
    lib.oracle_evaluate_chain.argtypes = [P, ctypes.c_int, i32p, i32p, i64p, i64p, i32p,
                                          ctypes.c_int, i64p, i64p, i64p]
    lib.oracle_free.argtypes = [P]
    lib.oracle_threads.restype = ctypes.c_int
    lib.oracle_threads.argtypes = []
    return lib


def _arr(xs, dtype):
    a = np.ascontiguousarray(np.asarray(xs, dtype=dtype))
    if a.size == 0:
        a = np.zeros(1, dtype=dtype)
    return a


def _ptr(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


class OracleResult:
    """Result of one oracle run; frees the C result when collected."""

    def __init__(self, graph, handle, lib):
        self._lib = lib
        self._h = handle
        self.graph = graph
        L = self._lib
        self.status = L.oracle_status(handle)
        self.num_sets = L.oracle_num_sets(handle)
        self.T_total = L.oracle_T_total(handle)
        self.num_pairs = L.oracle_num_pairs(handle)
        self.relaxations_literal = L.oracle_relaxations_literal(handle)
        self.t_star = L.oracle_t_star(handle)
        self.m_star = L.oracle_m_star(handle)
        self.k = L.oracle_k(handle)
        self.overhead = L.oracle_overhead(handle)
        self.peak = L.oracle_peak(handle)
        self.cache_mem = L.oracle_cache_mem(handle)

    def __del__(self):
        if getattr(self, "_h", None):
            self._lib.oracle_free(self._h)
            self._h = None

    @property
    def feasible(self):
        return self.status == OK

    def sets(self):
        """Family membership as a bool array [num_sets, n] in family order."""
        n = self.graph.n
        out = np.zeros((self.num_sets, max(n, 1)), dtype=np.uint8)
        if self.num_sets and n:
            self._lib.oracle_get_sets(self._h, out.ctypes.data)
        return out[:, :n].astype(bool)

    def rows(self, first=0, count=None):
        """opt and optarg rows [first, first+count); inf reads -1."""
        if count is None:
            count = self.num_sets - first
        W = self.T_total + 1
        opt = np.empty((count, W), dtype=np.int64)
        arg = np.empty((count, W), dtype=np.int32)
        if count:
            self._lib.oracle_get_rows(self._h, first, count, opt.ctypes.data, arg.ctypes.data)
        return opt, arg

    def table(self):
        return self.rows(0, self.num_sets)

    def schedule(self):
        """(chain family indices, seg[n], cached[n])."""
        n = self.graph.n
        chain = np.zeros(max(self.k, 1), dtype=np.int32)
        seg = np.zeros(max(n, 1), dtype=np.int32)
        cached = np.zeros(max(n, 1), dtype=np.uint8)
        self._lib.oracle_get_schedule(self._h, chain.ctypes.data, seg.ctypes.data, cached.ctypes.data)
        return chain[:self.k], seg[:n], cached[:n].astype(bool)

    def evaluate_chain(self, chain):
        """Eq. 1 overhead, Eq. 2 peak and M(U_k) of an arbitrary chain given
        as family indices (L_1..L_k)."""
        g = self.graph
        row_ptr, col_idx = g.csr()
        rp, ci = _arr(row_ptr, np.int32), _arr(col_idx, np.int32)
        T, M = _arr(g.T, np.int64), _arr(g.M, np.int64)
        ch = _arr(chain, np.int32)
        o, p, c = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        st = self._lib.oracle_evaluate_chain(self._h, g.n, _ptr(rp, ctypes.c_int32),
                                             _ptr(ci, ctypes.c_int32), _ptr(T, ctypes.c_int64),
                                             _ptr(M, ctypes.c_int64), _ptr(ch, ctypes.c_int32),
                                             len(chain), ctypes.byref(o), ctypes.byref(p),
                                             ctypes.byref(c))
        if st != OK:
            raise ValueError(f"oracle_evaluate_chain status {st}")
        return o.value, p.value, c.value


def solve(graph, mode, B, objective="tc", max_sets=1 << 20, max_sources=-1, csr=None,
          T=None, M=None, parallel=False):
    """Run the oracle.  ``graph`` is a workloads.Graph; ``csr``/``T``/``M``
    override its arrays (used to feed invalid inputs).  ``parallel`` runs the
    OpenMP build (same results, all cores)."""
    lib = _load(parallel)
    row_ptr, col_idx = csr if csr is not None else graph.csr()
    T = graph.T if T is None else T
    M = graph.M if M is None else M
    rp, ci = _arr(row_ptr, np.int32), _arr(col_idx, np.int32)
    Ta, Ma = _arr(T, np.int64), _arr(M, np.int64)
    h = lib.oracle_solve(graph.n, _ptr(rp, ctypes.c_int32), _ptr(ci, ctypes.c_int32),
                         _ptr(Ta, ctypes.c_int64), _ptr(Ma, ctypes.c_int64),
                         MODES[mode] if isinstance(mode, str) else mode, int(B),
                         OBJECTIVES[objective] if isinstance(objective, str) else objective,
                         int(max_sets), int(max_sources))
    if not h:
        raise MemoryError("oracle_solve returned NULL")
    return OracleResult(graph, h, lib)


def family(graph, mode, max_sets=1 << 20):
    """The lower-set family of Algorithm 1 only (no table): a result whose
    sets() and T_total are valid, in the family order of the solve."""
    lib = _load()
    row_ptr, col_idx = graph.csr()
    rp, ci = _arr(row_ptr, np.int32), _arr(col_idx, np.int32)
    Ta, Ma = _arr(graph.T, np.int64), _arr(graph.M, np.int64)
    h = lib.oracle_family(graph.n, _ptr(rp, ctypes.c_int32), _ptr(ci, ctypes.c_int32),
                          _ptr(Ta, ctypes.c_int64), _ptr(Ma, ctypes.c_int64),
                          MODES[mode] if isinstance(mode, str) else mode, int(max_sets))
    if not h:
        raise MemoryError("oracle_family returned NULL")
    return OracleResult(graph, h, lib)


def solve_dominance(graph, mode, B, max_sets=1 << 20, parallel=False):
    """Algorithm 1 with the dominance skip of Section 4.2's last paragraph
    (time-centric only): the same t* and opt[V, t*], a table whose entries
    are never below solve()'s."""
    lib = _load(parallel)
    row_ptr, col_idx = graph.csr()
    rp, ci = _arr(row_ptr, np.int32), _arr(col_idx, np.int32)
    Ta, Ma = _arr(graph.T, np.int64), _arr(graph.M, np.int64)
    h = lib.oracle_solve_dominance(graph.n, _ptr(rp, ctypes.c_int32), _ptr(ci, ctypes.c_int32),
                                   _ptr(Ta, ctypes.c_int64), _ptr(Ma, ctypes.c_int64),
                                   MODES[mode] if isinstance(mode, str) else mode, int(B),
                                   int(max_sets))
    if not h:
        raise MemoryError("oracle_solve_dominance returned NULL")
    return OracleResult(graph, h, lib)


def min_budget(graph, mode, parallel=False):
    """The smallest budget B for which the family admits a strategy.

    Section 5 runs its experiments at this budget and finds it by binary
    search.  Feasibility is monotone in B (a strategy whose peak is within B
    is within every larger budget) and B = 2 M(V) is always feasible (the
    one-segment chain {V} peaks at 2 M(V), Eq. 2), so bisection over
    [0, 2 M(V)] on whether Algorithm 1 finds a finite cell in row V gives it.
    """
    lo, hi = -1, 2 * int(sum(graph.M))
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if solve(graph, mode, mid, "tc", parallel=parallel).status == OK:
            hi = mid
        else:
            lo = mid
    return hi
