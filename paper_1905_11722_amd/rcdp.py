"""Python binding of the HIP library ``librcdp.so`` (argument marshalling only).

The names mirror the C ABI of ``include/rc.h``::

    g = Graph.create(workloads_graph)           # rc_graph_create
    fam = g.build_family("pruned")              # rc_build_family
    sol = fam.solve(B, "tc")                    # rc_solve
    sched = sol.reconstruct()                   # rc_reconstruct
    m, arg = sol.table()                        # rc_export_table

Device memory comes from PyTorch's caching allocator through the ABI's
allocator callbacks, and every call is enqueued on PyTorch's current HIP
stream.  There is no CPU fallback: without the compiled library, or
without a GPU, every entry point raises.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librcdp.so")

OK, INFEASIBLE = 0, 1
E_ARG, E_CYCLE, E_COST, E_TOO_MANY_SETS, E_OVERFLOW, E_NOMEM, E_DEVICE, E_STATE = (
    -1, -2, -3, -4, -5, -6, -7, -9)
E_SCRATCH = -10
MODES = {"exact": 0, "pruned": 1}
OBJECTIVES = {"tc": 0, "mc": 1}

ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p)
FREE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p)


class RcError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        detail = ""
        if status == E_DEVICE:
            detail = ": " + load_library().rc_last_error().decode(errors="replace")
        super().__init__(f"{where}: status {status} ({status_str(status)}){detail}")


class FamilyInfo(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("words", ctypes.c_int32), ("num_sets", ctypes.c_int64),
                ("num_pairs", ctypes.c_int64), ("num_levels", ctypes.c_int64),
                ("table_cells", ctypes.c_int64), ("relaxations", ctypes.c_int64),
                ("T_total", ctypes.c_int64), ("M_total", ctypes.c_int64),
                ("max_row", ctypes.c_int64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


_lib = None


def load_library():
    """Load ``librcdp.so``; raises ImportError when it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: run __graft_entry__.build() "
                          "(hipcc for gfx950) first; there is no fallback path")
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    pp = ctypes.POINTER(ctypes.c_void_p)
    lib.rc_status_str.restype = ctypes.c_char_p
    lib.rc_status_str.argtypes = [ctypes.c_int]
    lib.rc_last_error.restype = ctypes.c_char_p
    lib.rc_last_error.argtypes = []
    lib.rc_graph_create.restype = ctypes.c_int
    lib.rc_graph_create.argtypes = [i32, P, P, P, P, ALLOC_FN, FREE_FN, P, P, pp]
    lib.rc_graph_free.argtypes = [P]
    lib.rc_build_family.restype = ctypes.c_int
    lib.rc_build_family.argtypes = [P, i32, i64, P, pp]
    lib.rc_family_stats.restype = ctypes.c_int
    lib.rc_family_stats.argtypes = [P, ctypes.POINTER(FamilyInfo)]
    lib.rc_family_sets.restype = ctypes.c_int
    lib.rc_family_sets.argtypes = [P, P, P]
    lib.rc_family_free.argtypes = [P]
    lib.rc_solve.restype = ctypes.c_int
    lib.rc_solve.argtypes = [P, i64, i32, P, pp, ctypes.POINTER(i64), ctypes.POINTER(i64)]
    lib.rc_solve_dominance.restype = ctypes.c_int
    lib.rc_solve_dominance.argtypes = [P, i64, P, pp, ctypes.POINTER(i64), ctypes.POINTER(i64)]
    lib.rc_solution_fill_ms.restype = ctypes.c_int
    lib.rc_solution_fill_ms.argtypes = [P, ctypes.POINTER(ctypes.c_float)]
    lib.rc_solve_batch.restype = ctypes.c_int
    lib.rc_solve_batch.argtypes = [P, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.c_void_p]
    lib.rc_min_budget.restype = ctypes.c_int
    lib.rc_min_budget.argtypes = [P, ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64)]
    lib.rc_solve_dual.restype = ctypes.c_int
    lib.rc_solve_dual.argtypes = [P, i64, i32, P, ctypes.POINTER(i64), ctypes.POINTER(i64),
                                  ctypes.POINTER(ctypes.c_float), ctypes.POINTER(i32), P, P, P,
                                  ctypes.POINTER(i64), ctypes.POINTER(i64), ctypes.POINTER(i64)]
    lib.rc_solve_dual_noalloc.restype = ctypes.c_int
    lib.rc_solve_dual_noalloc.argtypes = [P, i64, i32, P, ctypes.POINTER(i64),
                                          ctypes.POINTER(i64), ctypes.POINTER(i32), P, P, P,
                                          ctypes.POINTER(i64), ctypes.POINTER(i64),
                                          ctypes.POINTER(i64)]
    lib.rc_solution_fill_kernel_ms.restype = ctypes.c_int
    lib.rc_solution_fill_kernel_ms.argtypes = [P, ctypes.POINTER(ctypes.c_float)]
    lib.rc_solution_fill_path.restype = ctypes.c_int
    lib.rc_solution_fill_path.argtypes = [P, ctypes.POINTER(ctypes.c_int32)]
    lib.rc_solution_trace_path.restype = ctypes.c_int
    lib.rc_solution_trace_path.argtypes = [P, ctypes.POINTER(ctypes.c_int32)]
    lib.rc_reconstruct.restype = ctypes.c_int
    lib.rc_reconstruct.argtypes = [P, P, ctypes.POINTER(i32), P, P, P, ctypes.POINTER(i64),
                                   ctypes.POINTER(i64), ctypes.POINTER(i64)]
    lib.rc_export_table.restype = ctypes.c_int
    lib.rc_export_table.argtypes = [P, i64, i64, P, P, P]
    lib.rc_solution_free.argtypes = [P]
    _lib = lib
    return lib


def status_str(status):
    return load_library().rc_status_str(status).decode()


def _check(status, where, allow=(OK,)):
    if status not in allow:
        raise RcError(status, where)
    return status


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


class _TorchAllocator:
    """Device memory from PyTorch's caching allocator (stream-ordered)."""

    def __init__(self):
        import torch
        self.torch = torch
        self.device = torch.cuda.current_device()
        self.alloc = ALLOC_FN(self._alloc)
        self.free = FREE_FN(self._free)

    def _alloc(self, nbytes, user):
        try:
            stream = self.torch.cuda.current_stream(self.device)
            return self.torch.cuda.caching_allocator_alloc(int(nbytes), self.device, stream)
        except Exception:  # noqa: BLE001 - report NULL to the C side
            return None

    def _free(self, ptr, user):
        self.torch.cuda.caching_allocator_delete(ptr)


_allocator = None


def _get_allocator():
    global _allocator
    if _allocator is None:
        _allocator = _TorchAllocator()
    return _allocator


def _i32(xs):
    a = np.ascontiguousarray(np.asarray(xs, dtype=np.int32))
    return a if a.size else np.zeros(1, dtype=np.int32)


@dataclass
class Schedule:
    """A traced chain and its Eq. 1 / Eq. 2 re-evaluation."""

    chain: np.ndarray      # family indices of L_1..L_k
    seg: np.ndarray        # 0-based segment of every node
    cached: np.ndarray     # bool, node in U_k
    overhead: int
    peak: int
    cache_mem: int


class Graph:
    """rc_graph: a validated DAG with costs, resident on the device."""

    def __init__(self, handle, n, keep):
        self._h = handle
        self.n = n
        self._keep = keep

    @classmethod
    def create(cls, graph=None, *, n=None, row_ptr=None, col_idx=None, T=None, M=None,
               allocator="torch"):
        lib = load_library()
        if graph is not None:
            n = graph.n
            row_ptr, col_idx = graph.csr()
            T, M = graph.T, graph.M
        rp, ci, Ta, Ma = _i32(row_ptr), _i32(col_idx), _i32(T), _i32(M)
        if allocator == "torch":
            al = _get_allocator()
            alloc, free = al.alloc, al.free
        else:
            alloc, free = ALLOC_FN(), FREE_FN()
        h = ctypes.c_void_p()
        st = lib.rc_graph_create(int(n), rp.ctypes.data, ci.ctypes.data, Ta.ctypes.data,
                                 Ma.ctypes.data, alloc, free, None, _stream(), ctypes.byref(h))
        _check(st, "rc_graph_create")
        return cls(h, int(n), (alloc, free))

    def build_family(self, mode, max_sets=65535):
        lib = load_library()
        h = ctypes.c_void_p()
        st = lib.rc_build_family(self._h, MODES.get(mode, mode), int(max_sets), _stream(),
                                 ctypes.byref(h))
        _check(st, "rc_build_family")
        return Family(h, self)

    def free(self):
        if self._h:
            load_library().rc_graph_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.free()
        except Exception:  # noqa: BLE001
            pass


class Family:
    """rc_family: the lower-set family and its pair data on the device."""

    def __init__(self, handle, graph):
        self._h = handle
        self.graph = graph
        info = FamilyInfo()
        _check(load_library().rc_family_stats(handle, ctypes.byref(info)), "rc_family_stats")
        self.info = info.as_dict()

    def sets(self):
        """Membership [num_sets, n] bool array in family order."""
        words = self.info["words"]
        F = self.info["num_sets"]
        buf = np.zeros((F, max(words, 1)), dtype=np.uint64)
        _check(load_library().rc_family_sets(self._h, buf.ctypes.data, _stream()), "rc_family_sets")
        n = self.graph.n
        out = np.zeros((F, n), dtype=bool)
        for v in range(n):
            out[:, v] = (buf[:, v // 64] >> np.uint64(v % 64)) & np.uint64(1)
        return out

    def min_budget(self):
        """The smallest budget with a strategy in this family (rc_min_budget)."""
        b = ctypes.c_int64(-1)
        _check(load_library().rc_min_budget(self._h, _stream(), ctypes.byref(b)), "rc_min_budget")
        return b.value

    def solve_dual(self, B, objective="tc", schedule=False):
        """(t, m, fill_ms) from the memory-indexed table (rc_solve_dual): t* and
        opt[V, t*] as rc_solve finds them, (-1, -1) when infeasible.  With
        schedule=True, (t, m, fill_ms, Schedule or None): the chain traced back
        through that table and its re-evaluated strategy."""
        lib = load_library()
        t, m, ms = ctypes.c_int64(-1), ctypes.c_int64(-1), ctypes.c_float(-1.0)
        if not schedule:
            st = lib.rc_solve_dual(self._h, int(B), OBJECTIVES.get(objective, objective),
                                   _stream(), ctypes.byref(t), ctypes.byref(m), ctypes.byref(ms),
                                   None, None, None, None, None, None, None)
            _check(st, "rc_solve_dual", allow=(OK, INFEASIBLE))
            return t.value, m.value, ms.value
        F = self.info["num_sets"]
        n = self.graph.n
        k = ctypes.c_int32(-1)
        chain = np.zeros(max(F, 1), dtype=np.int32)
        seg = np.zeros(max(n, 1), dtype=np.int32)
        cached = np.zeros(max(n, 1), dtype=np.uint8)
        o, p, c = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        st = lib.rc_solve_dual(self._h, int(B), OBJECTIVES.get(objective, objective), _stream(),
                               ctypes.byref(t), ctypes.byref(m), ctypes.byref(ms), ctypes.byref(k),
                               chain.ctypes.data, seg.ctypes.data, cached.ctypes.data,
                               ctypes.byref(o), ctypes.byref(p), ctypes.byref(c))
        _check(st, "rc_solve_dual", allow=(OK, INFEASIBLE))
        if st == INFEASIBLE:
            return t.value, m.value, ms.value, None
        return t.value, m.value, ms.value, Schedule(
            chain[:k.value].copy(), seg[:n].copy(), cached[:n].astype(bool), o.value, p.value,
            c.value)

    def solve_dual_noalloc(self, B, objective="tc"):
        """(t, m, Schedule or None) from rc_solve_dual_noalloc: the
        memory-indexed solve with its schedule, run in the library's static
        scratch instead of allocated memory."""
        lib = load_library()
        F = self.info["num_sets"]
        n = self.graph.n
        t, m, k = ctypes.c_int64(-1), ctypes.c_int64(-1), ctypes.c_int32(-1)
        chain = np.zeros(max(F, 1), dtype=np.int32)
        seg = np.zeros(max(n, 1), dtype=np.int32)
        cached = np.zeros(max(n, 1), dtype=np.uint8)
        o, p, c = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        st = lib.rc_solve_dual_noalloc(self._h, int(B), OBJECTIVES.get(objective, objective),
                                       _stream(), ctypes.byref(t), ctypes.byref(m),
                                       ctypes.byref(k), chain.ctypes.data, seg.ctypes.data,
                                       cached.ctypes.data, ctypes.byref(o), ctypes.byref(p),
                                       ctypes.byref(c))
        _check(st, "rc_solve_dual_noalloc", allow=(OK, INFEASIBLE))
        if st == INFEASIBLE:
            return t.value, m.value, None
        return t.value, m.value, Schedule(chain[:k.value].copy(), seg[:n].copy(),
                                          cached[:n].astype(bool), o.value, p.value, c.value)

    def sweep(self, budgets, objective="mc"):
        """Solve at every budget in one batched fill (rc_solve_batch):
        [(budget, Solution)].  The memory-centric sweep of Section 4.4 runs the
        same family at a range of budgets."""
        lib = load_library()
        Bs = np.asarray([int(B) for B in budgets], dtype=np.int64)
        nb = len(Bs)
        hs = (ctypes.c_void_p * nb)()
        t = np.full(nb, -1, dtype=np.int64)
        m = np.full(nb, -1, dtype=np.int64)
        st = lib.rc_solve_batch(self._h, Bs.ctypes.data, nb, OBJECTIVES.get(objective, objective),
                                _stream(), ctypes.cast(hs, ctypes.c_void_p), t.ctypes.data,
                                m.ctypes.data)
        _check(st, "rc_solve_batch")
        return [(int(Bs[b]), Solution(ctypes.c_void_p(hs[b]), self,
                                      OK if t[b] >= 0 else INFEASIBLE, int(t[b]), int(m[b])))
                for b in range(nb)]

    def solve(self, B, objective="tc"):
        lib = load_library()
        h = ctypes.c_void_p()
        t = ctypes.c_int64(-1)
        m = ctypes.c_int64(-1)
        st = lib.rc_solve(self._h, int(B), OBJECTIVES.get(objective, objective), _stream(),
                          ctypes.byref(h), ctypes.byref(t), ctypes.byref(m))
        _check(st, "rc_solve", allow=(OK, INFEASIBLE))
        return Solution(h, self, st, t.value, m.value)

    def solve_dominance(self, B):
        """rc_solve_dominance: the time-centric solve with the dominance skip;
        the table keeps each row's weak front, infinity elsewhere."""
        lib = load_library()
        h = ctypes.c_void_p()
        t = ctypes.c_int64(-1)
        m = ctypes.c_int64(-1)
        st = lib.rc_solve_dominance(self._h, int(B), _stream(), ctypes.byref(h), ctypes.byref(t),
                                    ctypes.byref(m))
        _check(st, "rc_solve_dominance", allow=(OK, INFEASIBLE))
        return Solution(h, self, st, t.value, m.value)

    def free(self):
        if self._h:
            load_library().rc_family_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.free()
        except Exception:  # noqa: BLE001
            pass


class Solution:
    """rc_solution: the DP table of one budget and its selected t*."""

    def __init__(self, handle, family, status, t_star, m_star):
        self._h = handle
        self.family = family
        self.status = status
        self.t_star = t_star
        self.m_star = m_star

    @property
    def feasible(self):
        return self.status == OK

    def fill_ms(self):
        ms = ctypes.c_float()
        _check(load_library().rc_solution_fill_ms(self._h, ctypes.byref(ms)), "rc_solution_fill_ms")
        return ms.value

    def fill_kernel_ms(self):
        ms = ctypes.c_float()
        _check(load_library().rc_solution_fill_kernel_ms(self._h, ctypes.byref(ms)),
               "rc_solution_fill_kernel_ms")
        return ms.value

    FILL_KERNELS = ("k_fill_level_vec", "k_fill_blocked", "k_fill_ghost", "k_fill_wide",
                    "k_fill_level")

    def fill_kernel(self):
        """Name of the fill kernel the solve ran (see rc_solution_fill_path)."""
        path = ctypes.c_int32()
        _check(load_library().rc_solution_fill_path(self._h, ctypes.byref(path)),
               "rc_solution_fill_path")
        return self.FILL_KERNELS[path.value]

    TRACE_KERNELS = ("k_trace", "k_trace_follow")

    def trace_kernel(self):
        """Name of the traceback kernel the last reconstruct ran, or None
        before the first (see rc_solution_trace_path)."""
        path = ctypes.c_int32()
        _check(load_library().rc_solution_trace_path(self._h, ctypes.byref(path)),
               "rc_solution_trace_path")
        return self.TRACE_KERNELS[path.value] if path.value >= 0 else None

    def reconstruct(self):
        lib = load_library()
        F = self.family.info["num_sets"]
        n = self.family.graph.n
        k = ctypes.c_int32()
        chain = np.zeros(max(F, 1), dtype=np.int32)
        seg = np.zeros(max(n, 1), dtype=np.int32)
        cached = np.zeros(max(n, 1), dtype=np.uint8)
        o, p, c = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        st = lib.rc_reconstruct(self._h, _stream(), ctypes.byref(k), chain.ctypes.data,
                                seg.ctypes.data, cached.ctypes.data, ctypes.byref(o),
                                ctypes.byref(p), ctypes.byref(c))
        _check(st, "rc_reconstruct")
        return Schedule(chain[:k.value].copy(), seg[:n].copy(), cached[:n].astype(bool),
                        o.value, p.value, c.value)

    def table(self, first=0, count=None):
        """Rows [first, first+count) over t = 0..T(V); -1 = infinite / none."""
        if count is None:
            count = self.family.info["num_sets"] - first
        W = self.family.info["T_total"] + 1
        m = np.empty((count, W), dtype=np.int64)
        a = np.empty((count, W), dtype=np.int32)
        st = load_library().rc_export_table(self._h, int(first), int(count), m.ctypes.data,
                                            a.ctypes.data, _stream())
        _check(st, "rc_export_table")
        return m, a

    def free(self):
        if self._h:
            load_library().rc_solution_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.free()
        except Exception:  # noqa: BLE001
            pass


def solve_graph(graph, mode, B, objective="tc"):
    """Convenience: build, solve and reconstruct one case."""
    g = Graph.create(graph)
    fam = g.build_family(mode)
    sol = fam.solve(B, objective)
    sched = sol.reconstruct() if sol.feasible else None
    return g, fam, sol, sched
