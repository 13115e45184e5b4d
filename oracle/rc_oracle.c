/*
 * rc_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded CPU implementation of the dynamic program
 * of Kusumoto et al., "A Graph Theoretic Framework of Recomputation
 * Algorithms for Memory-Efficient Backpropagation" (NeurIPS 2019):
 * the lower-set families of Sections 2 and 4.3, the canonical strategy's
 * overhead (Eq. 1) and peak memory (Eq. 2) of Section 3, and the DP of
 * Section 4.2 / Appendix A (Algorithm 1), with the memory-centric variant of
 * Section 4.4.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load this code.  The same source builds a single-threaded library and,
 * with OpenMP, an all-cores one whose tables are identical (the targets of
 * one source are split among threads; sources stay in order).  It shares
 * nothing with the GPU library: sets are plain
 * 0/1 byte arrays over the node ids, every set expression of Algorithm 1 is
 * formed explicitly for every (L, L') pair, and t runs over the whole range
 * 0..T(V) as printed.  Nothing is blocked, fused or reordered.
 *
 * Pins (see tests/test_oracle_*.py): brute force over every chain of the
 * family (the naive search of Section 4.1) for the whole opt table, the
 * optarg table and both objectives; the closed form of chain graphs; the
 * floor T(Sinks) and ceiling T(V) of the objectives; infeasibility below
 * 2 max M_v; monotonicity in B; pruned >= exact; the t-free row-minimum
 * DP; re-evaluation of the returned schedule with Eq. 1 / Eq. 2.  The
 * dominance skip (oracle_solve_dominance) against its closed form from the
 * brute-force table: every row keeps its weak front, and each cell is the
 * least one-step extension of the source rows' fronts.
 *
 * Readings of the paper taken here (each one is listed with its reason in
 * the design notes):
 *  - The pruned family {L^v} is completed with the empty set and V, which
 *    Algorithm 1 needs as its first and last keys.
 *  - Sets are visited in ascending size; equal sizes by ascending numeric
 *    value sum_{v in L} 2^v of the caller's node ids.  With the strict "<"
 *    update this makes optarg the smallest family index among equally good
 *    predecessors.
 *  - Terms (iii) and (iv) of Eq. 2 are added as printed, even where the two
 *    node sets overlap.
 *  - "Replacing min with max" for the memory-centric strategy changes only
 *    the selection of t in row V; the table is the same.
 *  - optarg keeps the predecessor's family index; its t is recovered as
 *    t' - T(V' \ boundary(L')).
 *  - The dominance skip (Section 4.2, last paragraph) compares each entry
 *    with the least of the same row's earlier entries, strictly, and is
 *    offered for the time-centric objective only.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_INFEASIBLE 1
#define ORC_E_ARG (-1)
#define ORC_E_CYCLE (-2)
#define ORC_E_COST (-3)
#define ORC_E_TOO_MANY_SETS (-4)
#define ORC_E_OVERFLOW (-5)
#define ORC_E_NOMEM (-6)
#define ORC_E_INTERNAL (-8)

#define INF INT64_MAX

typedef unsigned char u8;

/* The computation graph G = (V, E) of Section 2 with per-node costs. */
typedef struct {
  int n;
  u8* adj;          /* adj[v*n + w] = 1 iff (v, w) in E */
  int64_t* T;       /* forward time T_v > 0 */
  int64_t* M;       /* memory size M_v > 0 */
} graph;

typedef struct oracle_result {
  int status;
  int n;
  int64_t num_sets;
  int64_t T_total;  /* T(V) */
  u8* sets;         /* num_sets * n membership bytes, family order */
  int64_t* opt;     /* num_sets * (T_total + 1) */
  int32_t* arg;     /* same shape, -1 where no predecessor */
  int64_t num_pairs;
  int64_t relaxations_literal;  /* pairs * (T(V) + 1) */
  int64_t t_star;
  int64_t m_star;
  int32_t k;
  int32_t* chain;   /* family indices of L_1 .. L_k */
  int32_t* seg;     /* segment index (0-based) of every node */
  u8* cached;       /* 1 iff the node is in U_k */
  int64_t overhead; /* Eq. 1 of the returned chain */
  int64_t peak;     /* max_i of Eq. 2 of the returned chain */
  int64_t cache_mem;/* M(U_k) */
} oracle_result;

/* ---------------------------------------------------------------- sets */

/* T(S) and M(S) of Section 2: sums of the per-node costs over S. */
static int64_t cost_sum(int n, const u8* S, const int64_t* c) {
  int64_t s = 0;
  for (int v = 0; v < n; v++)
    if (S[v]) s += c[v];
  return s;
}

/* delta^+(S) of Section 2: nodes w with an edge (s, w) for some s in S. */
static void delta_plus(const graph* g, const u8* S, u8* out) {
  int n = g->n;
  for (int w = 0; w < n; w++) {
    out[w] = 0;
    for (int s = 0; s < n; s++)
      if (S[s] && g->adj[s * n + w]) { out[w] = 1; break; }
  }
}

/* delta^-(S) of Section 2: nodes v with an edge (v, s) for some s in S. */
static void delta_minus(const graph* g, const u8* S, u8* out) {
  int n = g->n;
  for (int v = 0; v < n; v++) {
    out[v] = 0;
    for (int s = 0; s < n; s++)
      if (S[s] && g->adj[v * n + s]) { out[v] = 1; break; }
  }
}

static void set_minus(int n, const u8* A, const u8* B, u8* out) {
  for (int v = 0; v < n; v++) out[v] = A[v] && !B[v];
}

static void set_and(int n, const u8* A, const u8* B, u8* out) {
  for (int v = 0; v < n; v++) out[v] = A[v] && B[v];
}

static void set_complement(int n, const u8* A, u8* out) {
  for (int v = 0; v < n; v++) out[v] = !A[v];
}

/* Boundary of L (Section 2): delta^-(V \ L) intersected with L. */
static void boundary(const graph* g, const u8* L, u8* out, u8* tmp) {
  int n = g->n;
  u8* comp = tmp;
  u8* dm = tmp + n;
  set_complement(n, L, comp);
  delta_minus(g, comp, dm);
  set_and(n, dm, L, out);
}

/* L proper subset of L2. */
static int proper_subset(int n, const u8* L, const u8* L2) {
  int strict = 0;
  for (int v = 0; v < n; v++) {
    if (L[v] && !L2[v]) return 0;
    if (!L[v] && L2[v]) strict = 1;
  }
  return strict;
}

/* -------------------------------------------------------------- family */

typedef struct {
  u8* sets;
  int64_t count;
  int64_t cap;
  int n;
  int overflow;
} family_buf;

static int family_push(family_buf* f, const u8* L) {
  if (f->count >= f->cap) { f->overflow = 1; return 0; }
  memcpy(f->sets + (size_t)f->count * f->n, L, (size_t)f->n);
  f->count++;
  return 1;
}

/* All lower sets (the exact family of Section 4.2): decide every node in a
 * topological order; a node may join only if all of its predecessors did,
 * which is exactly the condition delta^-(L) in L. */
static void enum_lower_sets(const graph* g, const int* topo, int pos, u8* cur,
                            family_buf* f) {
  int n = g->n;
  if (f->overflow) return;
  if (pos == n) { family_push(f, cur); return; }
  int v = topo[pos];
  enum_lower_sets(g, topo, pos + 1, cur, f);          /* v not in L */
  int ok = 1;
  for (int p = 0; p < n; p++)
    if (g->adj[p * n + v] && !cur[p]) { ok = 0; break; }
  if (ok) {                                           /* v in L */
    cur[v] = 1;
    enum_lower_sets(g, topo, pos + 1, cur, f);
    cur[v] = 0;
  }
}

/* L^v = { w : v is reachable from w } (Section 4.3): v and all ancestors. */
static void ancestor_set(const graph* g, int v, u8* out, int* stack) {
  int n = g->n, top = 0;
  memset(out, 0, (size_t)n);
  out[v] = 1;
  stack[top++] = v;
  while (top > 0) {
    int x = stack[--top];
    for (int p = 0; p < n; p++)
      if (g->adj[p * n + x] && !out[p]) { out[p] = 1; stack[top++] = p; }
  }
}

static int g_sort_n;
/* Family order: ascending |L|, then ascending sum_{v in L} 2^v. */
static int cmp_sets(const void* a, const void* b) {
  const u8* A = (const u8*)a;
  const u8* B = (const u8*)b;
  int n = g_sort_n, sa = 0, sb = 0;
  for (int v = 0; v < n; v++) { sa += A[v]; sb += B[v]; }
  if (sa != sb) return sa < sb ? -1 : 1;
  for (int v = n - 1; v >= 0; v--)
    if (A[v] != B[v]) return A[v] < B[v] ? -1 : 1;
  return 0;
}

/* ---------------------------------------------------------------- input */

static int build_graph(int n, const int32_t* row_ptr, const int32_t* col_idx,
                       const int64_t* T, const int64_t* M, graph* g, int* topo) {
  if (n < 0 || (n > 0 && (!row_ptr || !T || !M))) return ORC_E_ARG;
  g->n = n;
  g->adj = (u8*)calloc((size_t)n * n + 1, 1);
  g->T = (int64_t*)malloc(sizeof(int64_t) * (n + 1));
  g->M = (int64_t*)malloc(sizeof(int64_t) * (n + 1));
  if (!g->adj || !g->T || !g->M) return ORC_E_NOMEM;
  if (n == 0) return ORC_OK;
  if (row_ptr[0] != 0) return ORC_E_ARG;
  for (int v = 0; v < n; v++) {
    if (row_ptr[v + 1] < row_ptr[v]) return ORC_E_ARG;
    for (int e = row_ptr[v]; e < row_ptr[v + 1]; e++) {
      int w = col_idx[e];
      if (w < 0 || w >= n) return ORC_E_ARG;
      if (w == v) return ORC_E_CYCLE;
      g->adj[v * n + w] = 1;   /* E is a set: duplicates collapse */
    }
  }
  for (int v = 0; v < n; v++) {
    if (T[v] <= 0 || M[v] <= 0) return ORC_E_COST;   /* T_v, M_v > 0 */
    g->T[v] = T[v];
    g->M[v] = M[v];
  }
  /* topological order by repeatedly taking a node with no unplaced
   * predecessor; failure means a directed cycle */
  u8* placed = (u8*)calloc((size_t)n, 1);
  if (!placed) return ORC_E_NOMEM;
  for (int pos = 0; pos < n; pos++) {
    int found = -1;
    for (int v = 0; v < n && found < 0; v++) {
      if (placed[v]) continue;
      int ok = 1;
      for (int p = 0; p < n; p++)
        if (g->adj[p * n + v] && !placed[p]) { ok = 0; break; }
      if (ok) found = v;
    }
    if (found < 0) { free(placed); return ORC_E_CYCLE; }
    placed[found] = 1;
    topo[pos] = found;
  }
  free(placed);
  return ORC_OK;
}

/* ------------------------------------------------------------ Eq. 1 / 2 */

/* Overhead (Eq. 1) and peak memory (Eq. 2) of the canonical strategy of a
 * chain L_1 < ... < L_k = V, evaluated from the definitions of Section 3:
 * U_i is the union of the boundaries of L_1..L_i, the overhead is
 * T(V \ U_k), and segment i needs
 *   M(U_{i-1}) + 2 M(V_i) + M(delta+(L_i) \ L_i) + M(delta-(delta+(L_i)) \ L_i). */
static void evaluate_chain(const graph* g, const u8* sets, const int32_t* chain,
                           int k, int32_t* seg, u8* cached, int64_t* overhead,
                           int64_t* peak, int64_t* cache_mem) {
  int n = g->n;
  u8* U = (u8*)calloc((size_t)n + 1, 1);
  u8* prev = (u8*)calloc((size_t)n + 1, 1);
  u8* Vi = (u8*)calloc((size_t)n + 1, 1);
  u8* dp = (u8*)calloc((size_t)n + 1, 1);
  u8* dpo = (u8*)calloc((size_t)n + 1, 1);
  u8* dmdp = (u8*)calloc((size_t)n + 1, 1);
  u8* dmo = (u8*)calloc((size_t)n + 1, 1);
  u8* bd = (u8*)calloc((size_t)n + 1, 1);
  u8* tmp = (u8*)calloc((size_t)2 * n + 2, 1);
  int64_t pk = 0;
  for (int v = 0; v < n; v++) seg[v] = -1;
  for (int i = 0; i < k; i++) {
    const u8* Li = sets + (size_t)chain[i] * n;
    set_minus(n, Li, prev, Vi);
    for (int v = 0; v < n; v++)
      if (Vi[v]) seg[v] = i;
    delta_plus(g, Li, dp);
    set_minus(n, dp, Li, dpo);
    delta_minus(g, dp, dmdp);
    set_minus(n, dmdp, Li, dmo);
    int64_t mem = cost_sum(n, U, g->M) + 2 * cost_sum(n, Vi, g->M) +
                  cost_sum(n, dpo, g->M) + cost_sum(n, dmo, g->M);
    if (mem > pk) pk = mem;
    boundary(g, Li, bd, tmp);
    for (int v = 0; v < n; v++)
      if (bd[v]) U[v] = 1;                 /* U_i = U_{i-1} + boundary(L_i) */
    memcpy(prev, Li, (size_t)n);
  }
  u8* rest = (u8*)calloc((size_t)n + 1, 1);
  u8* all = (u8*)malloc((size_t)n + 1);
  memset(all, 1, (size_t)n + 1);
  set_minus(n, all, U, rest);
  *overhead = cost_sum(n, rest, g->T);
  *peak = pk;
  *cache_mem = cost_sum(n, U, g->M);
  for (int v = 0; v < n; v++) cached[v] = U[v];
  free(U); free(prev); free(Vi); free(dp); free(dpo); free(dmdp); free(dmo);
  free(bd); free(tmp); free(rest); free(all);
}

/* ----------------------------------------------------------------- DP */

void oracle_free(oracle_result* r);

/*
 * Algorithm 1 (Appendix A) over the family selected by mode (0: all lower
 * sets, Section 4.2; 1: {L^v} plus the empty set and V, Section 4.3).
 * objective 0 picks the smallest finite t in row V (time-centric); 1 the
 * largest (memory-centric, Section 4.4).  max_sources < 0 runs the whole
 * outer loop; otherwise only its first max_sources iterations (used to time
 * a bounded sample; the selection step is then skipped).
 */
static oracle_result* solve_impl(int n, const int32_t* row_ptr, const int32_t* col_idx,
                                 const int64_t* T, const int64_t* M, int mode, int64_t B,
                                 int objective, int64_t max_sets, int64_t max_sources,
                                 int dominance_skip, int family_only) {
  oracle_result* r = (oracle_result*)calloc(1, sizeof(oracle_result));
  if (!r) return NULL;
  r->n = n;
  r->t_star = -1;
  r->m_star = -1;
  graph g;
  memset(&g, 0, sizeof(g));
  int* topo = (int*)malloc(sizeof(int) * (n + 1));
  if (!topo) { r->status = ORC_E_NOMEM; return r; }
  int st = (mode != 0 && mode != 1) || B < 0 || (objective != 0 && objective != 1) ||
                   (dominance_skip && objective != 0)
               ? ORC_E_ARG : build_graph(n, row_ptr, col_idx, T, M, &g, topo);
  if (st != ORC_OK) { r->status = st; goto done; }

  /* ---- the family, in the order of Algorithm 1's outer loop ---- */
  {
    family_buf f;
    f.n = n > 0 ? n : 1;
    f.cap = max_sets;
    f.count = 0;
    f.overflow = 0;
    if (max_sets <= 0) { st = ORC_E_ARG; goto fail; }
    f.sets = (u8*)calloc((size_t)max_sets * f.n, 1);
    if (!f.sets) { st = ORC_E_NOMEM; goto fail; }
    f.n = n;
    u8* cur = (u8*)calloc((size_t)n + 1, 1);
    if (mode == 0) {
      enum_lower_sets(&g, topo, 0, cur, &f);
    } else {
      int* stack = (int*)malloc(sizeof(int) * (n + 1));
      u8* tmp = (u8*)calloc((size_t)n + 1, 1);
      family_push(&f, cur);                              /* empty set */
      for (int v = 0; v < n; v++) {
        ancestor_set(&g, v, tmp, stack);
        family_push(&f, tmp);
      }
      memset(tmp, 1, (size_t)n);                         /* V, if new */
      int have = 0;
      for (int64_t i = 0; i < f.count && n > 0; i++)
        if (memcmp(f.sets + (size_t)i * n, tmp, (size_t)n) == 0) have = 1;
      if (!have && n > 0) family_push(&f, tmp);
      free(stack);
      free(tmp);
    }
    free(cur);
    if (f.overflow) { free(f.sets); st = ORC_E_TOO_MANY_SETS; goto fail; }
    if (n > 0) {
      g_sort_n = n;
      qsort(f.sets, (size_t)f.count, (size_t)n, cmp_sets);
    }
    r->sets = f.sets;
    r->num_sets = f.count;
  }
  if (family_only) {
    for (int v = 0; v < n; v++) r->T_total += g.T[v];
    r->status = ORC_OK;
    goto done;
  }

  {
    const int64_t F = r->num_sets;
    int64_t TV = 0;
    for (int v = 0; v < n; v++) TV += g.T[v];          /* T(V) */
    r->T_total = TV;
    const int64_t W = TV + 1;
    if ((double)F * (double)W > 4.0e9) { st = ORC_E_OVERFLOW; goto fail; }
    r->opt = (int64_t*)malloc(sizeof(int64_t) * (size_t)(F * W));
    r->arg = (int32_t*)malloc(sizeof(int32_t) * (size_t)(F * W));
    if (!r->opt || !r->arg) { st = ORC_E_NOMEM; goto fail; }

    /* Init DP array: opt[L, t] = inf everywhere, opt[empty, 0] = 0. */
    for (int64_t x = 0; x < F * W; x++) { r->opt[x] = INF; r->arg[x] = -1; }
    r->opt[0] = 0;   /* family index 0 is the empty set */

    /* The set expressions of Algorithm 1 that involve L' alone are the same
     * for every L; they are formed once per family member:
     *   bd[L']  = boundary(L')
     *   out[L'] = M(delta+(L') \ L') + M(delta-(delta+(L')) \ L')       */
    u8* bdall = (u8*)calloc((size_t)F * (n > 0 ? n : 1), 1);
    int64_t* outm = (int64_t*)calloc((size_t)F, sizeof(int64_t));
    u8* dp = (u8*)calloc((size_t)n + 1, 1);
    u8* dpo = (u8*)calloc((size_t)n + 1, 1);
    u8* dmdp = (u8*)calloc((size_t)n + 1, 1);
    u8* dmo = (u8*)calloc((size_t)n + 1, 1);
    u8* tmp = (u8*)calloc((size_t)2 * n + 2, 1);
    if (!bdall || !outm || !dp || !dpo || !dmdp || !dmo || !tmp) { st = ORC_E_NOMEM; goto fail_loop; }
    for (int64_t j = 0; j < F; j++) {
      const u8* Lp = r->sets + (size_t)j * n;
      delta_plus(&g, Lp, dp);
      set_minus(n, dp, Lp, dpo);
      delta_minus(&g, dp, dmdp);
      set_minus(n, dmdp, Lp, dmo);
      outm[j] = cost_sum(n, dpo, g.M) + cost_sum(n, dmo, g.M);
      boundary(&g, Lp, bdall + (size_t)j * n, tmp);
    }

    const int64_t sources = max_sources < 0 ? F : (max_sources < F ? max_sources : F);
    int64_t pairs = 0, literal = 0;
    int err = ORC_OK;
    /* Built with OpenMP (the all-cores timing build), the targets L' of one
     * source L are shared among threads: each thread owns whole rows L',
     * and L still advances in family order, so every cell sees its updates
     * in the order of the sequential loop and ends with the same value and
     * optarg.  Built without it, the pragmas are ignored. */
#pragma omp parallel reduction(+ : pairs, literal)
    {
      u8* Vp = (u8*)calloc((size_t)n + 1, 1);
      u8* Vpb = (u8*)calloc((size_t)n + 1, 1);
      u8* bdl = (u8*)calloc((size_t)n + 1, 1);
      if (!Vp || !Vpb || !bdl) {
#pragma omp atomic write
        err = ORC_E_NOMEM;
      }
      /* for L in the family in ascending order of size */
      for (int64_t i = 0; i < sources; i++) {
        const u8* L = r->sets + (size_t)i * n;
        /* for L' in the family with L a proper subset of L' */
#pragma omp for schedule(dynamic, 4)
        for (int64_t j = 0; j < F; j++) {
          if (!Vp || !Vpb || !bdl) continue;
          const u8* Lp = r->sets + (size_t)j * n;
          if (!proper_subset(n, L, Lp)) continue;
          pairs++;
          literal += TV + 1;
          const u8* bd = bdall + (size_t)j * n;
          /* V' = L' \ L */
          set_minus(n, Lp, L, Vp);
          /* 2 M(V') + M(delta+(L') \ L') + M(delta-(delta+(L')) \ L') */
          const int64_t mem_terms = 2 * cost_sum(n, Vp, g.M) + outm[j];
          /* T(V' \ boundary(L')) and M(boundary(L') \ L) */
          set_minus(n, Vp, bd, Vpb);
          const int64_t dT = cost_sum(n, Vpb, g.T);
          set_minus(n, bd, L, bdl);
          const int64_t dM = cost_sum(n, bdl, g.M);
          /* for t = 0..T(V) */
          const int64_t* optL = r->opt + (size_t)(i * W);
          int64_t* optLp = r->opt + (size_t)(j * W);
          int32_t* argLp = r->arg + (size_t)(j * W);
          int64_t least = INF;                /* min of opt[L, u] over u < t */
          for (int64_t t = 0; t <= TV; t++) {
            const int64_t m = optL[t];
            if (m == INF) continue;
            /* the skip of Section 4.2 (last paragraph): an earlier t of the
             * same row with strictly less memory makes this entry useless */
            const int dominated = dominance_skip && least < m;
            if (m < least) least = m;
            if (dominated) continue;
            const int64_t Mcal = m + mem_terms;
            if (Mcal > B) continue;             /* memory constraint */
            const int64_t tp = t + dT;
            const int64_t mp = m + dM;
            if (tp > TV) {
#pragma omp atomic write
              err = ORC_E_INTERNAL;
              break;
            }
            if (optLp[tp] > mp) {               /* update DP array */
              optLp[tp] = mp;
              argLp[tp] = (int32_t)i;
            }
          }
        }
      }
      free(Vp); free(Vpb); free(bdl);
    }
    r->num_pairs = pairs;
    r->relaxations_literal = literal;
    if (err != ORC_OK) st = err;
  fail_loop:
    free(dp); free(dpo); free(dmdp); free(dmo);
    free(tmp); free(bdall); free(outm);
    if (st != ORC_OK) goto fail;
    if (max_sources >= 0) { r->status = ORC_OK; goto done; }

    /* ---- selection: t* = min (time-centric) or max (memory-centric) of
     *      the finite entries of row V ---- */
    const int64_t* optV = r->opt + (size_t)((F - 1) * W);
    int64_t ts = -1;
    for (int64_t t = 0; t <= TV; t++) {
      if (optV[t] == INF) continue;
      if (ts < 0 || objective == 1) ts = t;
      if (objective == 0) break;
    }
    if (ts < 0) { r->status = ORC_INFEASIBLE; goto done; }
    r->t_star = ts;
    r->m_star = optV[ts];

    /* ---- traceback of optarg from (V, t*) ---- */
    int32_t* rev = (int32_t*)malloc(sizeof(int32_t) * (size_t)(F + 1));
    u8* bd2 = (u8*)calloc((size_t)n + 1, 1);
    u8* vp2 = (u8*)calloc((size_t)n + 1, 1);
    u8* vpb2 = (u8*)calloc((size_t)n + 1, 1);
    u8* tmp2 = (u8*)calloc((size_t)2 * n + 2, 1);
    int64_t j = F - 1, t = ts;
    int k = 0;
    while (j != 0) {
      int32_t i = r->arg[(size_t)(j * W + t)];
      if (i < 0 || k > F) { st = ORC_E_INTERNAL; break; }
      const u8* L = r->sets + (size_t)i * n;
      const u8* Lp = r->sets + (size_t)j * n;
      set_minus(n, Lp, L, vp2);
      boundary(&g, Lp, bd2, tmp2);
      set_minus(n, vp2, bd2, vpb2);
      t -= cost_sum(n, vpb2, g.T);
      rev[k++] = (int32_t)j;
      j = i;
    }
    if (st == ORC_OK && t != 0) st = ORC_E_INTERNAL;   /* must end at (empty, 0) */
    free(bd2); free(vp2); free(vpb2); free(tmp2);
    if (st != ORC_OK) { free(rev); goto fail; }
    r->k = k;
    r->chain = (int32_t*)malloc(sizeof(int32_t) * (size_t)(k + 1));
    for (int x = 0; x < k; x++) r->chain[x] = rev[k - 1 - x];
    free(rev);
    r->seg = (int32_t*)malloc(sizeof(int32_t) * (size_t)(n + 1));
    r->cached = (u8*)calloc((size_t)n + 1, 1);
    evaluate_chain(&g, r->sets, r->chain, k, r->seg, r->cached, &r->overhead, &r->peak,
                   &r->cache_mem);
    r->status = ORC_OK;
    goto done;
  }

fail:
  r->status = st;
done:
  free(topo);
  free(g.adj);
  free(g.T);
  free(g.M);
  return r;
}

oracle_result* oracle_solve(int n, const int32_t* row_ptr, const int32_t* col_idx,
                            const int64_t* T, const int64_t* M, int mode, int64_t B,
                            int objective, int64_t max_sets, int64_t max_sources) {
  return solve_impl(n, row_ptr, col_idx, T, M, mode, B, objective, max_sets, max_sources, 0, 0);
}

/* The family of Algorithm 1 alone (mode as oracle_solve), in its order, with
 * no table: oracle_get_sets and oracle_T_total are valid on the result. */
oracle_result* oracle_family(int n, const int32_t* row_ptr, const int32_t* col_idx,
                             const int64_t* T, const int64_t* M, int mode, int64_t max_sets) {
  return solve_impl(n, row_ptr, col_idx, T, M, mode, 0, 0, max_sets, -1, 0, 1);
}

/*
 * Algorithm 1 with the skip of Section 4.2's last paragraph: when t < t'
 * and opt[L, t] < opt[L, t'], the entry opt[L, t'] is not propagated.  Any
 * chain through (L, t') is matched by the same continuation from (L, t),
 * faster and within the budget, so the time-centric t* and opt[V, t*] are
 * unchanged while other entries may grow; only objective 0 is accepted.
 */
oracle_result* oracle_solve_dominance(int n, const int32_t* row_ptr, const int32_t* col_idx,
                                      const int64_t* T, const int64_t* M, int mode, int64_t B,
                                      int64_t max_sets) {
  return solve_impl(n, row_ptr, col_idx, T, M, mode, B, 0, max_sets, -1, 1, 0);
}

/* ---------------------------------------------------------- accessors */

/* Threads the fill loop runs on: 1 unless built with OpenMP. */
int oracle_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

int oracle_status(const oracle_result* r) { return r->status; }
int64_t oracle_num_sets(const oracle_result* r) { return r->num_sets; }
int64_t oracle_T_total(const oracle_result* r) { return r->T_total; }
int64_t oracle_num_pairs(const oracle_result* r) { return r->num_pairs; }
int64_t oracle_relaxations_literal(const oracle_result* r) { return r->relaxations_literal; }
int64_t oracle_t_star(const oracle_result* r) { return r->t_star; }
int64_t oracle_m_star(const oracle_result* r) { return r->m_star; }
int32_t oracle_k(const oracle_result* r) { return r->k; }
int64_t oracle_overhead(const oracle_result* r) { return r->overhead; }
int64_t oracle_peak(const oracle_result* r) { return r->peak; }
int64_t oracle_cache_mem(const oracle_result* r) { return r->cache_mem; }

/* Membership bytes of the family, num_sets * n, in family order. */
void oracle_get_sets(const oracle_result* r, u8* out) {
  if (r->sets) memcpy(out, r->sets, (size_t)r->num_sets * (size_t)r->n);
}

/* Rows [first, first+count) of the table; infinite entries read -1. */
void oracle_get_rows(const oracle_result* r, int64_t first, int64_t count, int64_t* opt,
                     int32_t* arg) {
  const int64_t W = r->T_total + 1;
  for (int64_t x = 0; x < count * W; x++) {
    int64_t v = r->opt[(size_t)(first * W + x)];
    if (opt) opt[x] = v == INF ? -1 : v;
    if (arg) arg[x] = r->arg[(size_t)(first * W + x)];
  }
}

void oracle_get_schedule(const oracle_result* r, int32_t* chain, int32_t* seg, u8* cached) {
  if (chain && r->chain) memcpy(chain, r->chain, sizeof(int32_t) * (size_t)r->k);
  if (seg && r->seg) memcpy(seg, r->seg, sizeof(int32_t) * (size_t)r->n);
  if (cached && r->cached) memcpy(cached, r->cached, (size_t)r->n);
}

/* Eq. 1 / Eq. 2 of an arbitrary chain given as family indices. */
int oracle_evaluate_chain(const oracle_result* r, int n, const int32_t* row_ptr,
                          const int32_t* col_idx, const int64_t* T, const int64_t* M,
                          const int32_t* chain, int k, int64_t* overhead, int64_t* peak,
                          int64_t* cache_mem) {
  graph g;
  memset(&g, 0, sizeof(g));
  int* topo = (int*)malloc(sizeof(int) * (n + 1));
  int st = build_graph(n, row_ptr, col_idx, T, M, &g, topo);
  if (st == ORC_OK) {
    int32_t* seg = (int32_t*)malloc(sizeof(int32_t) * (n + 1));
    u8* cached = (u8*)malloc((size_t)n + 1);
    evaluate_chain(&g, r->sets, chain, k, seg, cached, overhead, peak, cache_mem);
    free(seg);
    free(cached);
  }
  free(topo); free(g.adj); free(g.T); free(g.M);
  return st;
}

void oracle_free(oracle_result* r) {
  if (!r) return;
  free(r->sets);
  free(r->opt);
  free(r->arg);
  free(r->chain);
  free(r->seg);
  free(r->cached);
  free(r);
}
