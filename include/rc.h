/*
 * rc.h -- C ABI of the MI355X solver for the General Recomputation Problem
 * of Kusumoto et al., "A Graph Theoretic Framework of Recomputation
 * Algorithms for Memory-Efficient Backpropagation" (NeurIPS 2019).
 *
 * Problem (Section 3, definition of the General Recomputation Problem):
 * given the computation DAG G = (V, E) of a network with per-node forward
 * time T_v > 0 and memory size M_v > 0 (Section 2), and a memory budget B,
 * find an increasing chain of lower sets L_1 < ... < L_k = V whose
 * canonical strategy has the least recomputation overhead (Eq. 1) among
 * those whose peak memory (Eq. 2) is at most B, or report that none exists.
 * The solver is the dynamic program of Section 4.2 / Appendix A (Algorithm
 * 1) over either the family of all lower sets (Section 4.2) or the pruned
 * family of ancestor sets (Section 4.3), with the time-centric (minimum
 * overhead) or memory-centric (maximum overhead, Section 4.4) selection.
 *
 * Life cycle:  rc_graph_create -> rc_build_family -> rc_solve ->
 * rc_reconstruct / rc_export_table -> rc_solution_free -> rc_family_free
 * -> rc_graph_free.  A handle must outlive every handle made from it.
 *
 * Conventions shared by every entry point:
 *  - Every pointer argument named *_host is host memory owned by the caller;
 *    the library copies what it needs and keeps no caller pointer.
 *  - Device memory comes from the caller's allocator (alloc/free_fn/user of
 *    rc_graph_create), or from hipMalloc/hipFree when alloc is NULL.  Each
 *    handle owns the device buffers it allocated and releases them in its
 *    *_free call.
 *  - stream is a hipStream_t (NULL: the default stream).  Device work is
 *    enqueued on it; entry points that return results to the host
 *    synchronise that stream before returning.
 *  - A negative return is an error: out-parameters are left untouched and
 *    no handle is created.  RC_INFEASIBLE is a result, not an error.
 *    Nothing crosses the ABI as an exception.
 *  - Handles are not thread-safe; distinct handles may be used from
 *    distinct threads.
 *  - Node ids 0..n-1 are the caller's.  They fix the order of sets of equal
 *    size (ascending numeric value sum_{v in L} 2^v), and through it which of
 *    several equally good predecessors the traceback follows (the smallest
 *    family index, as with the strict update of Algorithm 1).
 *
 * Environment switches (read when a family is built or a table is solved;
 * none changes a result, only which kernels compute it and how they are
 * shaped; an unrecognised value is ignored):
 *  - RCDP_FILL = level | wavefront | wide | ghost: the fill of Algorithm 1.
 *    level: one launch per group of equal-size sets (k_fill_level_vec on
 *    16-bit cells, k_fill_level on 32-bit cells).
 *    wavefront: the persistent row-push wavefront over fixed blocks of
 *    targets (k_fill_blocked).  wide: the split-panel wavefront over fixed
 *    blocks (k_fill_wide).  ghost: the wavefront over ghost-zone blocks
 *    (k_fill_ghost; families of at most 4096 sets).  Unset: chosen from the
 *    family's size, width and number of levels (rc_solution_fill_path
 *    reports the choice).
 *  - RCDP_WIDE_NP = 1 | 2 | 3 | 4: panel waves per workgroup of
 *    k_fill_wide (default 3, or 1 for a launch of more columns than fit on
 *    the GPU at once with three: batched sweeps and the widest tables).
 *  - RCDP_CPT = 1 | 2 | 4: cells per thread of a k_fill_blocked column
 *    (default from the table's width).
 *  - RCDP_GHOST_CPT = 1 | 2: cells per thread of a k_fill_ghost column
 *    (default from the table's width).
 *  - RCDP_DEBUG (any value): the wavefront fills print their launch shape
 *    to stderr.
 *  - RCDP_TRACE = scan | slice: the traceback of rc_reconstruct (see
 *    rc_solution_trace_path).  Unset: the slice when its (t* + 1) P pair
 *    tests (P the family's pairs) number at most 2^26 and at most 4e5 per
 *    step of the longest possible chain (min(num_sets - 1, n) steps), and
 *    its 4 (t* + 1) num_sets bytes at most 64 MiB; slice forces it within
 *    that size.
 *  - RCDP_JITTER = n (a nonzero integer): the race test.  The persistent
 *    wavefront fills (k_fill_blocked, k_fill_wide, k_fill_ghost) make their
 *    waves sleep pseudo-random times drawn from n at block starts and
 *    before a column publishes its progress, so that columns interleave in
 *    orders a plain run seldom takes; slower, same results.
 */
#ifndef RC_H
#define RC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct rc_graph_s* rc_graph;       /* validated DAG, device-resident */
typedef struct rc_family_s* rc_family;     /* lower-set family + pair data  */
typedef struct rc_solution_s* rc_solution; /* DP table of one budget        */

/* Device allocator: returns device memory of at least `bytes` bytes aligned
 * to 256 bytes, or NULL.  free_fn releases a pointer returned by alloc. */
typedef void* (*rc_alloc_fn)(size_t bytes, void* user);
typedef void (*rc_free_fn)(void* ptr, void* user);

enum rc_mode { RC_FAMILY_EXACT = 0, RC_FAMILY_PRUNED = 1 };
enum rc_objective { RC_TIME_CENTRIC = 0, RC_MEMORY_CENTRIC = 1 };

enum rc_status {
  RC_OK = 0,
  RC_INFEASIBLE = 1,        /* no chain meets the budget (a result) */
  RC_E_ARG = -1,            /* bad argument: NULL, out of range, bad CSR */
  RC_E_CYCLE = -2,          /* G has a directed cycle or a self-loop */
  RC_E_COST = -3,           /* some T_v or M_v is not positive */
  RC_E_TOO_MANY_SETS = -4,  /* the family exceeds max_sets or 65535 */
  RC_E_OVERFLOW = -5,       /* a value exceeds the table's integer widths */
  RC_E_NOMEM = -6,          /* the allocator returned NULL */
  RC_E_DEVICE = -7,         /* a HIP call failed or a kernel reported an error */
  RC_E_STATE = -9,          /* the handle is in the wrong state for the call */
  RC_E_SCRATCH = -10        /* the allocation-free entry point's scratch is too small */
};

/* Family statistics (rc_family_info).
 *  relaxations: the DP's unit of work, one (L, L', t) of Algorithm 1's
 *  update loop (Appendix A) whose source opt[L, t] can be finite: the sum
 *  over predecessor pairs (L, L') of w_L = T(L \ boundary(L)) + 1, since a
 *  chain ending at L recomputes only nodes of L \ boundary(L) (Eq. 1
 *  charges V_i \ boundary(L_i) per segment), so opt[L, t] is infinite for
 *  larger t.  Section 4.2's complexity O(T(V) #F^2) counts the same loop
 *  over every t.
 *  table_cells: sum over the family of w_L. */
typedef struct {
  int32_t n;            /* nodes */
  int32_t words;        /* 64-bit words per set bitmask, ceil(n / 64) */
  int64_t num_sets;     /* family size, including the empty set and V */
  int64_t num_pairs;    /* pairs L proper subset of L', both in the family */
  int64_t num_levels;   /* distinct set sizes (the DP's sequential steps) */
  int64_t table_cells;
  int64_t relaxations;
  int64_t T_total;      /* T(V) */
  int64_t M_total;      /* M(V) */
  int64_t max_row;      /* max_L w_L */
} rc_family_info;

/*
 * rc_graph_create -- validate G and its costs (Section 2) and copy them to
 * the device.
 *  n: number of nodes (0 allowed: then V is empty and the only chain is empty).
 *  row_ptr_host[n+1], col_idx_host[row_ptr[n]]: successor lists in CSR form;
 *    an entry w in row v is the edge (v, w), v directly needed to compute w.
 *    row_ptr[0] == 0 and non-decreasing.  Duplicate edges are ignored.
 *  T_host[n], M_host[n]: forward time and memory size, each >= 1.
 *  alloc/free_fn/user: device allocator used by this graph and by every
 *    family and solution made from it (NULL alloc: hipMalloc).
 * Errors: RC_E_ARG (NULL pointer, n < 0, n > 4096, index out of range,
 * row_ptr not monotone), RC_E_CYCLE (cycle or self-loop), RC_E_COST
 * (T_v or M_v < 1), RC_E_OVERFLOW (T(V) >= 2^31 - 1 or M(V) >= 2^31 / 4),
 * RC_E_NOMEM, RC_E_DEVICE.
 */
int rc_graph_create(int32_t n, const int32_t* row_ptr_host, const int32_t* col_idx_host,
                    const int32_t* T_host, const int32_t* M_host, rc_alloc_fn alloc,
                    rc_free_fn free_fn, void* user, void* stream, rc_graph* out);
void rc_graph_free(rc_graph g);

/*
 * rc_build_family -- build the lower-set family of Algorithm 1 on the
 * device, with every per-set and per-pair quantity the DP needs.
 *  mode RC_FAMILY_EXACT: all lower sets L (delta^-(L) in L, Section 2),
 *    the family of the exact DP (Section 4.2).
 *  mode RC_FAMILY_PRUNED: L^v = {w : v reachable from w} for every v
 *    (Section 4.3), plus the empty set and V, which the DP starts from and
 *    ends at.
 *  Sets are ordered by ascending size, then ascending numeric value; index
 *  0 is the empty set and index num_sets-1 is V.
 *  max_sets: cap on the family size (at most 65535).
 * The family does not depend on B: one family serves any number of solves.
 * Errors: RC_E_ARG, RC_E_TOO_MANY_SETS, RC_E_OVERFLOW (table cells or pairs
 * beyond 2^40), RC_E_NOMEM, RC_E_DEVICE.
 */
int rc_build_family(rc_graph g, int32_t mode, int64_t max_sets, void* stream, rc_family* out);
int rc_family_stats(rc_family f, rc_family_info* info);
/* Family members as bitmasks: bits_host[s * words + w] holds nodes
 * 64w..64w+63 of set s (bit v % 64), s in family order. */
int rc_family_sets(rc_family f, uint64_t* bits_host, void* stream);
/*
 * rc_min_budget -- the smallest budget B for which the family admits a
 * strategy (Section 5 runs its experiments at this budget and finds it by
 * binary search).  Computed on the device: B is feasible exactly when the
 * t-free form of Algorithm 1 (f[empty] = 0, f[L'] = min of f[L] + dm over the
 * pairs L < L' with f[L] + c(L, L') <= B; the row minima of the opt table)
 * reaches V, feasibility is monotone in B, and B = 2 M(V) is always feasible,
 * so the search runs over [0, 2 M(V)] with 64 budgets per round.
 *  *B_min: that budget (rc_solve(f, *B_min, ...) is feasible, *B_min - 1 is
 *  not).  Synchronises stream.
 * Returns RC_OK, RC_E_ARG (NULL argument), RC_E_OVERFLOW (2 M(V) >= 2^31 - 1),
 * RC_E_NOMEM, RC_E_DEVICE.
 */
int rc_min_budget(rc_family f, void* stream, int64_t* B_min);
/*
 * rc_solve_dual -- t* and opt[V, t*] of rc_solve, and a schedule attaining
 * them, from a table indexed by cached memory instead of time.  Algorithm 1
 * (Section 4.2, Appendix A) moves a chain state (L, t, m) along a pair
 * L < L' to (L', t + dt, m + dm) when m + c <= B, a test on m alone; this
 * table keeps, per (L, m) with m in [0, min(B, M(V))], the least t
 * (RC_TIME_CENTRIC) or the greatest t (RC_MEMORY_CENTRIC, Section 4.4) over
 * the chains reaching that state.  Its rows have min(B, M(V)) + 1 cells
 * instead of T(L \ boundary(L)) + 1, and its optimum over row V equals
 * rc_solve's: *t_opt = t*, *m_opt = the least m attaining it = opt[V, t*]
 * (both -1 when infeasible).
 *  B >= 0 as rc_solve.  *fill_ms (may be NULL): milliseconds between HIP
 *  events around the table's kernels.
 *  Schedule (computed only if one of these is non-NULL and B is feasible):
 *  the chain traced back through the table -- from (V, m*, t*) the smallest
 *  family index L whose cell (L, m - dm) passes the budget test and holds
 *  t - dt -- re-evaluated from Section 3's definitions; *k, chain_host[num
 *  sets], seg_host[n], cached_host[n], *overhead (Eq. 1, = t*), *peak (Eq. 2,
 *  <= B), *cache_mem (M(U_k) = opt[V, t*]) as rc_reconstruct.  Among equally
 *  good chains it may pick another than rc_reconstruct.
 *  Synchronises stream; device memory comes from the family's allocator and
 *  is returned before the call ends.
 * Returns RC_OK, RC_INFEASIBLE, or RC_E_ARG (NULL family, B < 0, bad
 * objective), RC_E_OVERFLOW (T(V) >= 2^32 - 1, or more than 2^31 cells),
 * RC_E_NOMEM, RC_E_DEVICE.
 */
int rc_solve_dual(rc_family f, int64_t B, int32_t objective, void* stream, int64_t* t_opt,
                  int64_t* m_opt, float* fill_ms, int32_t* k, int32_t* chain_host,
                  int32_t* seg_host, uint8_t* cached_host, int64_t* overhead, int64_t* peak,
                  int64_t* cache_mem);
/*
 * rc_solve_dual_noalloc -- rc_solve_dual without any allocation, for callers
 * that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  It calls no hipMalloc,
 * hipFree, event creation or allocating routine; the table, the status block
 * and the schedule buffers live in a file-scope device array of 16 MiB that
 * every GPU the library runs on holds until the process ends.  The family
 * (built beforehand with rc_build_family) and the host outputs are the
 * caller's, as with rc_solve_dual.
 *  Arguments, outputs and results as rc_solve_dual (no fill_ms).  The
 *  scratch takes 256 + 4 (num_sets + n) + n bytes plus the table's
 *  num_sets * (min(B, 2 M(V), M(V)) + 1) * 4 bytes, each part rounded up to
 *  256 bytes; a larger solve returns RC_E_SCRATCH and does nothing.
 *  Calls on one GPU share its scratch: calls that overlap on one GPU (other
 *  threads or streams) race and must be serialised by the caller.
 * Returns RC_OK, RC_INFEASIBLE, RC_E_ARG, RC_E_OVERFLOW, RC_E_SCRATCH,
 * RC_E_DEVICE.
 */
int rc_solve_dual_noalloc(rc_family f, int64_t B, int32_t objective, void* stream,
                          int64_t* t_opt, int64_t* m_opt, int32_t* k, int32_t* chain_host,
                          int32_t* seg_host, uint8_t* cached_host, int64_t* overhead,
                          int64_t* peak, int64_t* cache_mem);
void rc_family_free(rc_family f);

/*
 * rc_solve -- fill the DP table opt[L, t] (Section 4.2: the least cache
 * memory M(U_i) over chains ending at L with overhead t whose segments all
 * fit B) and select t* (Algorithm 1's final step).
 *  B >= 0: memory budget in the units of M.  Budgets above 2 M(V) give the
 *    same table as B = 2 M(V), since no segment of Eq. 2 exceeds 2 M(V).
 *  objective RC_TIME_CENTRIC: t* = min{t : opt[V, t] finite};
 *    RC_MEMORY_CENTRIC: t* = max{t : opt[V, t] finite} (Section 4.4).
 *  *t_opt, *m_opt: t* and opt[V, t*], or -1 and -1 when infeasible.
 * Cells are 16 bits wide while min(B, 2 M(V)) <= 65532 (every fill path);
 * above that the table takes 32-bit cells and the one-launch-per-level fill
 * (rc_solution_fill_path reports 4), with the same results.
 * Returns RC_OK or RC_INFEASIBLE (both create *out, whose table can be
 * exported), or an error: RC_E_ARG, RC_E_OVERFLOW (min(B, 2 M(V)) > 2^30,
 * which rc_graph_create's limit on M(V) rules out), RC_E_NOMEM, RC_E_DEVICE.
 */
int rc_solve(rc_family f, int64_t B, int32_t objective, void* stream, rc_solution* out,
             int64_t* t_opt, int64_t* m_opt);
/*
 * rc_solve_dominance -- rc_solve (time-centric) with the skip of Section
 * 4.2's last paragraph: a cell opt[L, t'] is not propagated when some t < t'
 * of the same row has opt[L, t] < opt[L, t'].  The table is filled one size
 * level at a time; once a level is done, each of its rows keeps only its
 * weak front (the cells whose m is no larger than every earlier cell of the
 * row) and stores every other cell as infinity, and later levels read no
 * source cell past the end of that front.
 *  t* and opt[V, t*] equal rc_solve's.  The exported table holds, at every
 *  front cell, the value of Algorithm 1 run with the skip (it is the same
 *  front as rc_solve's table), infinity elsewhere; the optarg of a front
 *  cell and the schedule of rc_reconstruct follow Algorithm 1 with the skip
 *  (the smallest family index among the sources that are propagated).
 *  Other arguments, handles and errors as rc_solve, except that the skip
 *  takes 16-bit cells only: RC_E_OVERFLOW when min(B, 2 M(V)) > 65532.
 */
int rc_solve_dominance(rc_family f, int64_t B, void* stream, rc_solution* out, int64_t* t_opt,
                       int64_t* m_opt);
/*
 * rc_solve_batch -- rc_solve at nb budgets of one family in one pass: the
 * memory-centric sweep of Section 4.4 solves the same family at a range of
 * budgets.  The tables are filled together (for wide tables one launch of
 * the wavefront kernel hands out the columns of all nb tables), then each
 * is selected as rc_solve would.
 *  B_host[nb]: budgets (>= 0).  out_host[nb]: one solution handle per
 *  budget, each freed with rc_solution_free.  t_opt[nb], m_opt[nb] (may be
 *  NULL): as rc_solve, -1 where infeasible.
 *  rc_solution_fill_ms / rc_solution_fill_kernel_ms of every handle report
 *  the time of the whole batched fill.
 * Returns RC_OK (every budget solved, feasible or not), or an error as
 * rc_solve (then no handle is created): RC_E_ARG (NULL, nb <= 0, a negative
 * budget, bad objective), RC_E_OVERFLOW, RC_E_NOMEM, RC_E_DEVICE.
 */
int rc_solve_batch(rc_family f, const int64_t* B_host, int32_t nb, int32_t objective,
                   void* stream, rc_solution* out_host, int64_t* t_opt, int64_t* m_opt);
/* Milliseconds between HIP events recorded on the solve's stream just
 * before the first and just after the last DP-fill kernel of the solve. */
int rc_solution_fill_ms(rc_solution s, float* ms);
/* Milliseconds between HIP events recorded on the solve's stream just
 * before and just after the one wavefront kernel of the blocked fill
 * (without the kernels that prepare its records).  On the level path,
 * which runs one launch per group of equal-size sets, this equals
 * rc_solution_fill_ms.  Returns RC_OK or RC_E_ARG (NULL argument). */
int rc_solution_fill_kernel_ms(rc_solution s, float* ms);
/* Which fill the solve ran (all of them compute the same table, Algorithm 1
 * of Section 4.2): *path = 0 one launch per group of equal-size sets on
 * 16-bit cells (k_fill_level_vec), 1 the persistent row-push wavefront
 * (k_fill_blocked), 2 the ghost-zone wavefront (k_fill_ghost), 3 the
 * split-panel wavefront (k_fill_wide), 4 one launch per group of equal-size
 * sets on 32-bit cells (k_fill_level).  Returns RC_OK or RC_E_ARG (NULL
 * argument). */
int rc_solution_fill_path(rc_solution s, int32_t* path);
/* Which traceback the last rc_reconstruct of the handle ran (both follow
 * the optarg rule of Section 4.2 and give the same chain): *path = 0 a
 * scan of the predecessor list at every step (k_trace), 1 optarg of every
 * cell (L', t') with t' <= t* evaluated at once, then followed
 * (k_trace_args, k_trace_follow); -1 before the first rc_reconstruct.
 * Returns RC_OK or RC_E_ARG (NULL argument). */
int rc_solution_trace_path(rc_solution s, int32_t* path);

/*
 * rc_reconstruct -- trace optarg back from (V, t*) (Section 4.2) and
 * re-evaluate the resulting canonical strategy from its definition.
 *  *k: chain length; chain_host[num_sets] (first *k used): family indices of
 *    L_1 .. L_k (L_k = V).
 *  seg_host[n]: 0-based index i of the segment V_{i+1} holding each node.
 *  cached_host[n]: 1 iff the node is in U_k = union of boundary(L_i).
 *  *overhead: Eq. 1, T(V \ U_k) (equals t*).  *peak: max_i of Eq. 2 (at
 *  most B).  *cache_mem: M(U_k) (equals opt[V, t*]).
 * Any of the output pointers may be NULL.
 * Returns RC_OK, RC_INFEASIBLE (nothing written), RC_E_ARG, RC_E_DEVICE.
 */
int rc_reconstruct(rc_solution s, void* stream, int32_t* k, int32_t* chain_host,
                   int32_t* seg_host, uint8_t* cached_host, int64_t* overhead,
                   int64_t* peak, int64_t* cache_mem);

/*
 * rc_export_table -- copy rows [first_set, first_set + num_sets) of the
 * table to the host, over the whole range t = 0..T(V) of Algorithm 1:
 * m_host[r * (T(V)+1) + t] = opt[L, t] (-1 when infinite) and
 * arg_host[...] = family index of optarg[L, t] (-1 when none).  Either
 * output may be NULL.  Returns RC_OK, RC_E_ARG, RC_E_NOMEM, RC_E_DEVICE.
 */
int rc_export_table(rc_solution s, int64_t first_set, int64_t num_sets, int64_t* m_host,
                    int32_t* arg_host, void* stream);
void rc_solution_free(rc_solution s);

/* Static description of a status code. */
const char* rc_status_str(int status);
/* Description of the last RC_E_DEVICE returned on the calling thread (the
 * failing HIP call and its error string, or the kernel-reported condition);
 * empty when none.  Valid until the next call on that thread. */
const char* rc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RC_H */
