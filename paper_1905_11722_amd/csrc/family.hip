// Graph encoding and lower-set family construction on the device.
//
// Sets of nodes are bitmasks of `words` 64-bit words (node v is bit v % 64
// of word v / 64).  Per-set work runs one wavefront per set with lane w
// holding word w (at most 64 words, i.e. 4096 nodes), so unions,
// differences and subset tests are single VALU ops per lane and set sums
// are lane-local popcount-style loops followed by a wave reduction.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "rc_internal.h"

namespace rcdp {

namespace {

constexpr int kWave = 64;

__device__ __forceinline__ int64_t wave_sum_i64(int64_t x) {
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, kWave);
  return x;
}

__device__ __forceinline__ uint64_t bcast_u64(uint64_t x, int lane) {
  return __shfl(x, lane, kWave);
}

// Sum of c[v] over the set bits of one word (nodes 64*word + bit).
__device__ __forceinline__ int64_t word_cost(uint64_t bits, int word, const int32_t* c) {
  int64_t s = 0;
  while (bits) {
    const int b = __builtin_ctzll(bits);
    s += c[word * 64 + b];
    bits &= bits - 1;
  }
  return s;
}

// ---------------------------------------------------------------- graph

// Gathers up to kPackMax device segments (whole 32-bit words) into one
// buffer, so that the results a host call reads back cost one copy; block
// row y copies segment y.
__global__ __launch_bounds__(256) void k_pack(PackList L, uint32_t* dst) {
  if ((int)blockIdx.y >= L.n) return;
  const PackSeg sg = L.seg[blockIdx.y];
  const uint32_t* src = static_cast<const uint32_t*>(sg.src);
  uint32_t* out = dst + sg.dst_off / 4;
  const int64_t words = sg.bytes / 4;
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < words;
       x += (int64_t)gridDim.x * blockDim.x)
    out[x] = src[x];
}

__global__ void k_zero_u64(uint64_t* p, int64_t count) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

// Edge (v, w): bit w in succ[v], bit v in pred[w] (Section 2's delta sets
// of single nodes).  Duplicate edges OR the same bit.
__global__ void k_graph_masks(int n, int words, const int32_t* row_ptr, const int32_t* col_idx,
                              uint64_t* succ, uint64_t* pred) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= n) return;
  for (int e = row_ptr[v]; e < row_ptr[v + 1]; e++) {
    const int w = col_idx[e];
    atomicOr((unsigned long long*)&succ[(int64_t)v * words + (w >> 6)], 1ull << (w & 63));
    atomicOr((unsigned long long*)&pred[(int64_t)w * words + (v >> 6)], 1ull << (v & 63));
  }
}

// ------------------------------------------------------------- ancestors

// L^v = {w : v reachable from w} (Section 4.3) = {v} + union of L^p over the
// predecessors p of v.  Nodes are visited depth by depth (longest path from
// a source), so every predecessor is final before it is read.  One
// workgroup; the closure lives in LDS when it fits.
template <bool kLds>
__global__ __launch_bounds__(1024) void k_ancestors(int n, int words, int num_depths,
                                                    int num_edges, const int32_t* by_depth,
                                                    const int32_t* depth_ptr,
                                                    const int32_t* pred_ptr,
                                                    const int32_t* pred_idx, uint64_t* anc_out) {
  // LDS variant: the ancestor masks, the depth order and the predecessor
  // lists all live in LDS, so each depth costs LDS traffic and one barrier
  extern __shared__ uint64_t lds_anc[];
  uint64_t* anc = kLds ? lds_anc : anc_out;
  int32_t* l_pp = reinterpret_cast<int32_t*>(lds_anc + (kLds ? (int64_t)n * words : 0));
  int32_t* l_pi = l_pp + (n + 1);
  int32_t* l_bd = l_pi + num_edges;
  int32_t* l_dp = l_bd + n;
  if (kLds) {
    for (int x = threadIdx.x; x <= n; x += blockDim.x) l_pp[x] = pred_ptr[x];
    for (int x = threadIdx.x; x < num_edges; x += blockDim.x) l_pi[x] = pred_idx[x];
    for (int x = threadIdx.x; x < n; x += blockDim.x) l_bd[x] = by_depth[x];
    for (int x = threadIdx.x; x <= num_depths; x += blockDim.x) l_dp[x] = depth_ptr[x];
    __syncthreads();
  }
  const int32_t* PP = kLds ? l_pp : pred_ptr;
  const int32_t* PI = kLds ? l_pi : pred_idx;
  const int32_t* BD = kLds ? l_bd : by_depth;
  const int32_t* DP = kLds ? l_dp : depth_ptr;
  for (int d = 0; d < num_depths; d++) {
    const int b = DP[d], e = DP[d + 1];
    const int items = (e - b) * words;
    for (int it = threadIdx.x; it < items; it += blockDim.x) {
      const int v = BD[b + it / words];
      const int w = it % words;
      uint64_t x = (v >> 6) == w ? (1ull << (v & 63)) : 0ull;
      for (int q = PP[v]; q < PP[v + 1]; q++) x |= anc[(int64_t)PI[q] * words + w];
      anc[(int64_t)v * words + w] = x;
    }
    __syncthreads();
  }
  if (kLds) {
    for (int it = threadIdx.x; it < n * words; it += blockDim.x) anc_out[it] = anc[it];
  }
}

// Small graphs: one wave walks the nodes in depth order (a topological
// order) with the masks, the depth order and the predecessor lists in LDS;
// lane w owns word w of every mask.  A node's predecessors are all earlier
// in the order, and one wave's LDS accesses complete in order, so the walk
// needs no barrier at all (the depth-parallel sweep pays one per depth).
__global__ __launch_bounds__(64) void k_ancestors_wave(int n, int words, int num_edges,
                                                       const int32_t* by_depth,
                                                       const int32_t* pred_ptr,
                                                       const int32_t* pred_idx,
                                                       uint64_t* anc_out) {
  extern __shared__ uint64_t lds_anc[];
  uint64_t* anc = lds_anc;
  int32_t* l_pp = reinterpret_cast<int32_t*>(lds_anc + (int64_t)n * words);
  int32_t* l_pi = l_pp + (n + 1);
  int32_t* l_bd = l_pi + num_edges;
  const int lane = threadIdx.x;
  for (int x = lane; x <= n; x += kWave) l_pp[x] = pred_ptr[x];
  for (int x = lane; x < num_edges; x += kWave) l_pi[x] = pred_idx[x];
  for (int x = lane; x < n; x += kWave) l_bd[x] = by_depth[x];
  __syncthreads();
  const bool active = lane < words;
  if (n == 0) return;
  int v = l_bd[0];
  int q0 = l_pp[v], q1 = l_pp[v + 1];
  for (int idx = 0; idx < n; idx++) {
    const int vn = idx + 1 < n ? l_bd[idx + 1] : v;     // the next node, ahead
    uint64_t x = (v >> 6) == lane ? (1ull << (v & 63)) : 0ull;
    int q = q0;
    for (; q + 4 <= q1; q += 4) {
      const int a0 = l_pi[q], a1 = l_pi[q + 1], a2 = l_pi[q + 2], a3 = l_pi[q + 3];
      if (active)
        x |= anc[(int64_t)a0 * words + lane] | anc[(int64_t)a1 * words + lane] |
             anc[(int64_t)a2 * words + lane] | anc[(int64_t)a3 * words + lane];
    }
    for (; q < q1; q++)
      if (active) x |= anc[(int64_t)l_pi[q] * words + lane];
    if (active) anc[(int64_t)v * words + lane] = x;
    q0 = l_pp[vn];
    q1 = l_pp[vn + 1];
    v = vn;
  }
  __syncthreads();
  for (int it = lane; it < n * words; it += kWave) anc_out[it] = anc[it];
}

// Transitive closure of the predecessor relation in one workgroup (graphs
// whose masks fit LDS and have at most kClosureWords words): A[v] starts as
// the direct predecessors of v; for every node k, each mask that contains k
// absorbs A[k] (Warshall's algorithm, any order of k).  A[k] never contains
// k in a DAG, so the bit tests of step k read values that step k does not
// change.  One barrier per node, every (node, word) item of a step in
// parallel; then L^v = A[v] + {v}.
constexpr int kClosureWords = 8;
constexpr int kClosureThreads = 1024;
constexpr int kClosureItems = 4;        // items per thread: n * words <= 4096

__global__ __launch_bounds__(kClosureThreads) void k_ancestors_closure(int n, int words,
                                                                       const uint64_t* pred_mask,
                                                                       uint64_t* anc_out) {
  extern __shared__ uint64_t A[];
  const int items = n * words;
  for (int x = threadIdx.x; x < items; x += kClosureThreads) A[x] = pred_mask[x];
  int vw[kClosureItems], wo[kClosureItems];          // row offset v * words and word w
#pragma unroll
  for (int r = 0; r < kClosureItems; r++) {
    const int it = threadIdx.x + r * kClosureThreads;
    const int v = it / words;
    vw[r] = it < items ? v * words : -1;
    wo[r] = it - v * words;
  }
  __syncthreads();
  for (int k = 0; k < n; k++) {
    const int kw = k >> 6;
    const uint64_t kb = 1ull << (k & 63);
    const int kr = k * words;
#pragma unroll
    for (int r = 0; r < kClosureItems; r++) {
      if (vw[r] < 0) continue;
      if (A[vw[r] + kw] & kb) A[vw[r] + wo[r]] |= A[kr + wo[r]];
    }
    __syncthreads();
  }
  for (int x = threadIdx.x; x < items; x += kClosureThreads) {
    const int v = x / words, w = x - v * words;
    anc_out[x] = A[x] | ((v >> 6) == w ? 1ull << (v & 63) : 0ull);
  }
}

// Candidates of the pruned family, set-major: [0] = empty set,
// [1 + v] = L^v, [n + 1] = V.
__global__ void k_pruned_candidates(int n, int words, const uint64_t* anc, uint64_t* cand) {
  const int64_t total = (int64_t)(n + 2) * words;
  for (int64_t it = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; it < total;
       it += (int64_t)gridDim.x * blockDim.x) {
    const int64_t c = it / words;
    const int w = (int)(it % words);
    uint64_t x;
    if (c == 0) {
      x = 0;
    } else if (c <= n) {
      x = anc[(c - 1) * words + w];
    } else {
      const int lo = w * 64;
      const int cnt = n - lo;
      x = cnt >= 64 ? ~0ull : ((1ull << cnt) - 1);
    }
    cand[it] = x;
  }
}

// ---------------------------------------------------- exact enumeration

// One size level of reverse search over lower sets.  A lower set X != {}
// has the canonical parent X \ {x}, x the largest node id of X with no
// successor inside X (removing such an x keeps delta^-(X \ {x}) inside).
// For every parent P of size s and node v with v not in P and
// delta^-(v) inside P, the child X = P + {v} is kept iff v is X's
// canonical element: every node of P with a larger id has a successor in X
// (v itself has none: a successor of v inside P would put v in P).
// Children are appended through an atomic counter; their order within the
// level is fixed afterwards by the rank kernel.
__global__ __launch_bounds__(256) void k_enum_level(int n, int words, int s, const uint64_t* succ,
                                                    const uint64_t* pred, uint64_t* cand,
                                                    int64_t cap, int32_t* lvl, DevStatus* st) {
  const int64_t pb = lvl[s], pe = lvl[s + 1];
  const int64_t items = (pe - pb) * n;
  for (int64_t it = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; it < items;
       it += (int64_t)gridDim.x * blockDim.x) {
    const int64_t p = pb + it / n;
    const int v = (int)(it % n);
    const uint64_t* P = cand + p * words;
    const int vw = v >> 6;
    const uint64_t vb = 1ull << (v & 63);
    if (P[vw] & vb) continue;
    bool ok = true;
    for (int w = 0; w < words && ok; w++) ok = (pred[(int64_t)v * words + w] & ~P[w]) == 0;
    if (!ok) continue;
    // every x in P with x > v needs a successor in X = P + {v}
    for (int w = words - 1; w >= vw && ok; w--) {
      uint64_t bits = P[w];
      if (w == vw) bits &= ~((vb << 1) - 1);  // ids > v only
      while (bits && ok) {
        const int x = w * 64 + __builtin_ctzll(bits);
        bits &= bits - 1;
        bool has = false;
        for (int u = 0; u < words && !has; u++) {
          uint64_t X = P[u] | (u == vw ? vb : 0ull);
          has = (succ[(int64_t)x * words + u] & X) != 0;
        }
        ok = has;
      }
    }
    if (!ok) continue;
    const unsigned long long slot = atomicAdd((unsigned long long*)&st->count, 1ull);
    if ((int64_t)slot >= cap) {
      st->overflow = 1;
      continue;
    }
    for (int w = 0; w < words; w++) cand[(int64_t)slot * words + w] = P[w] | (w == vw ? vb : 0ull);
  }
}

__global__ void k_enum_start(int words, uint64_t* cand, int32_t* lvl, DevStatus* st) {
  for (int w = threadIdx.x; w < words; w += blockDim.x) cand[w] = 0;  // the empty set
  if (threadIdx.x == 0) {
    st->count = 1;
    st->overflow = 0;
    lvl[0] = 0;
    lvl[1] = 1;
  }
}

// After level s: sets of size s + 1 occupy [lvl[s+1], count).
__global__ void k_enum_close(int s, int64_t cap, int32_t* lvl, DevStatus* st) {
  const int64_t c = st->count;
  lvl[s + 2] = (int32_t)(c < cap ? c : cap);
}

// --------------------------------------------------------------- ranking

// Numeric comparison of two sets stored set-major (most significant word
// first): -1, 0, 1.
__device__ __forceinline__ int cmp_value(const uint64_t* a, const uint64_t* b, int words) {
  for (int w = words - 1; w >= 0; w--)
    if (a[w] != b[w]) return a[w] < b[w] ? -1 : 1;
  return 0;
}

__device__ __forceinline__ int popcnt_set(const uint64_t* a, int words) {
  int c = 0;
  for (int w = 0; w < words; w++) c += __popcll(a[w]);
  return c;
}

// Canonical order: ascending size, then ascending numeric value.  Exact
// family: candidates are grouped by size level (reverse search yields no
// duplicates) and ranked within their level.  Output is word-major:
// bits[w * fstride + index].
__global__ __launch_bounds__(256) void k_rank(int words, int n, const uint64_t* cand,
                                              const int32_t* lvl, uint64_t* bits, int64_t fstride,
                                              DevStatus* st) {
  const int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  const int64_t total = lvl[n + 1];
  if (x >= total) return;
  const uint64_t* X = cand + x * words;
  const int s = popcnt_set(X, words);
  int64_t rank = lvl[s];
  for (int64_t y = lvl[s]; y < lvl[s + 1]; y++)
    if (y != x && cmp_value(cand + y * words, X, words) < 0) rank++;
  if (x == 0) st->count = st->overflow ? st->count : total;
  if (rank >= fstride) {
    st->error = 1;
    return;
  }
  for (int w = 0; w < words; w++) bits[(int64_t)w * fstride + rank] = X[w];
}

// Pruned family: candidates are [0] the empty set, [1..n] the sets L^v
// (pairwise distinct), [n+1] V, which is dropped when some L^v already
// equals V.  One workgroup: the candidates are bucketed by size (a counting
// sort in LDS), and a candidate's index is the number of candidates of
// smaller size plus those of its own size with a smaller numeric value.
__global__ __launch_bounds__(1024) void k_rank_pruned(int words, int n, const uint64_t* cand,
                                                      uint64_t* bits, int64_t fstride,
                                                      DevStatus* st) {
  constexpr int kThreads = 1024;
  __shared__ int32_t s_sz[kMaxNodes + 2];
  __shared__ int32_t s_start[kMaxNodes + 2];   // candidates of size < s, s = 0..n+1
  __shared__ int32_t s_next[kMaxNodes + 2];    // next free slot of each size's bucket
  __shared__ int32_t s_list[kMaxNodes + 2];    // candidates grouped by size
  __shared__ int32_t s_wsum[kThreads / kWave];
  __shared__ int32_t s_vdup;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  const int total = n + 2, bins = n + 2;       // sizes 0..n, counted one bin up
  if (tid == 0) s_vdup = n == 0;                 // V is the empty set itself
  for (int x = tid; x < bins; x += kThreads) s_start[x] = 0;
  for (int x = tid; x < total; x += kThreads) s_sz[x] = popcnt_set(cand + (int64_t)x * words, words);
  __syncthreads();
  for (int x = 1 + tid; x <= n; x += kThreads)
    if (s_sz[x] == n) s_vdup = 1;                 // some L^v is V already
  __syncthreads();
  const int valid = s_vdup ? n + 1 : n + 2;
  for (int x = tid; x < valid; x += kThreads) atomicAdd(&s_start[s_sz[x] + 1], 1);
  __syncthreads();
  // inclusive scan of the counts: s_start[s] = candidates of size < s
  const int per = (bins + kThreads - 1) / kThreads;
  const int b0 = min(bins, tid * per), b1 = min(bins, b0 + per);
  int run = 0;
  for (int q = b0; q < b1; q++) {
    run += s_start[q];
    s_start[q] = run;
  }
  int incl = run;
  for (int off = 1; off < kWave; off <<= 1) {
    const int y = __shfl_up(incl, off, kWave);
    if (lane >= off) incl += y;
  }
  if (lane == kWave - 1) s_wsum[wave] = incl;
  __syncthreads();
  int before = incl - run;
  for (int q = 0; q < wave; q++) before += s_wsum[q];
  for (int q = b0; q < b1; q++) {
    s_start[q] += before;
    s_next[q] = s_start[q];
  }
  __syncthreads();
  for (int x = tid; x < valid; x += kThreads) s_list[atomicAdd(&s_next[s_sz[x]], 1)] = x;
  __syncthreads();
  for (int x = tid; x < valid; x += kThreads) {
    const uint64_t* X = cand + (int64_t)x * words;
    const int sx = s_sz[x];
    int64_t rank = s_start[sx];
    for (int q = s_start[sx]; q < s_start[sx + 1]; q++) {
      const int y = s_list[q];
      if (y != x && cmp_value(cand + (int64_t)y * words, X, words) < 0) rank++;
    }
    if (rank >= fstride) {
      st->error = 1;
      continue;
    }
    for (int w = 0; w < words; w++) bits[(int64_t)w * fstride + rank] = X[w];
  }
  if (tid == 0) st->count = valid;
}

// ------------------------------------------------------- per-set values

// Per set L (one wave, lane w = word w):
//   boundary(L) = {v in L : some successor of v outside L}  (Section 2)
//   T(L), M(L), T(boundary), M(boundary)
//   A(L) = M(delta+(L) \ L) + M(delta-(delta+(L) \ L) \ L), the terms (iii)
//   and (iv) of Eq. 2 for the set L' = L (for a lower set L the
//   predecessors of delta+(L) inside L add nothing outside L)
//   w_L = T(L \ boundary(L)) + 1, the cells of row L that can be finite.
template <bool kLds>
__global__ __launch_bounds__(256) void k_set_quantities(
    int64_t F, int n, int words, int64_t fstride, const uint64_t* bits, const uint64_t* succ_g,
    const uint64_t* pred_g, const int32_t* T, const int32_t* M, uint64_t* bd, int32_t* size,
    int32_t* Tsum, int32_t* Msum, int32_t* Tbd, int32_t* Mbd, int32_t* A, int32_t* w_out) {
  // small graphs: the successor and predecessor masks of every node in LDS
  extern __shared__ uint64_t lds_nb[];
  const uint64_t* succ = succ_g;
  const uint64_t* pred = pred_g;
  if (kLds) {
    const int64_t cnt = (int64_t)n * words;
    for (int64_t x = threadIdx.x; x < cnt; x += blockDim.x) {
      lds_nb[x] = succ_g[x];
      lds_nb[cnt + x] = pred_g[x];
    }
    __syncthreads();
    succ = lds_nb;
    pred = lds_nb + cnt;
  }
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t s = blockIdx.x * (int64_t)(blockDim.x / kWave) + threadIdx.x / kWave;
  if (s >= F) return;
  const bool active = lane < words;
  const uint64_t L = active ? bits[(int64_t)lane * fstride + s] : 0ull;
  uint64_t out = 0, bdw = 0;
  for (int ww = 0; ww < words; ww++) {
    uint64_t Lw = bcast_u64(L, ww);
    while (Lw) {
      const int v = ww * 64 + __builtin_ctzll(Lw);
      Lw &= Lw - 1;
      const uint64_t sv = active ? succ[(int64_t)v * words + lane] : 0ull;
      out |= sv;
      const bool leaves = __any((sv & ~L) != 0);
      if (leaves && lane == ww) bdw |= 1ull << (v & 63);
    }
  }
  out &= ~L;
  uint64_t in2 = 0;
  for (int ww = 0; ww < words; ww++) {
    uint64_t Ow = bcast_u64(out, ww);
    while (Ow) {
      const int v = ww * 64 + __builtin_ctzll(Ow);
      Ow &= Ow - 1;
      if (active) in2 |= pred[(int64_t)v * words + lane];
    }
  }
  in2 &= ~L;
  const int64_t tl = wave_sum_i64(active ? word_cost(L, lane, T) : 0);
  const int64_t ml = wave_sum_i64(active ? word_cost(L, lane, M) : 0);
  const int64_t tb = wave_sum_i64(active ? word_cost(bdw, lane, T) : 0);
  const int64_t mb = wave_sum_i64(active ? word_cost(bdw, lane, M) : 0);
  const int64_t ao = wave_sum_i64(active ? word_cost(out, lane, M) : 0);
  const int64_t ai = wave_sum_i64(active ? word_cost(in2, lane, M) : 0);
  const int sz = (int)wave_sum_i64(active ? __popcll(L) : 0);
  if (active) bd[(int64_t)lane * fstride + s] = bdw;
  if (lane == 0) {
    size[s] = sz;
    Tsum[s] = (int32_t)tl;
    Msum[s] = (int32_t)ml;
    Tbd[s] = (int32_t)tb;
    Mbd[s] = (int32_t)mb;
    A[s] = (int32_t)(ao + ai);
    w_out[s] = (int32_t)(tl - tb + 1);
  }
}

// The same quantities for graphs of at most kLaneWords * 64 nodes, with the
// nodes spread over the lanes instead of walked one by one: lane l takes
// node 64 ww + l of every word ww, ORs its successor (then predecessor)
// words into kLaneWords register accumulators and adds its costs; word w
// of a union is then one wave OR reduction, a sum one wave sum.
constexpr int kLaneWords = 8;

__device__ __forceinline__ uint64_t readlane_u64(uint64_t x, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)x, l);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(x >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_or_u64(uint64_t x) {
  for (int off = 32; off > 0; off >>= 1) x |= __shfl_xor(x, off, kWave);
  return x;
}

template <bool kLds>
__global__ __launch_bounds__(256) void k_set_quantities_lanes(
    int64_t F, int n, int words, int64_t fstride, const uint64_t* bits, const uint64_t* succ_g,
    const uint64_t* pred_g, const int32_t* T, const int32_t* M, uint64_t* bd, int32_t* size,
    int32_t* Tsum, int32_t* Msum, int32_t* Tbd, int32_t* Mbd, int32_t* A, int32_t* w_out) {
  extern __shared__ uint64_t lds_nb[];
  const uint64_t* succ = succ_g;
  const uint64_t* pred = pred_g;
  if (kLds) {
    const int64_t cnt = (int64_t)n * words;
    for (int64_t x = threadIdx.x; x < cnt; x += blockDim.x) {
      lds_nb[x] = succ_g[x];
      lds_nb[cnt + x] = pred_g[x];
    }
    __syncthreads();
    succ = lds_nb;
    pred = lds_nb + cnt;
  }
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t s = blockIdx.x * (int64_t)(blockDim.x / kWave) + threadIdx.x / kWave;
  if (s >= F) return;
  // word w of L on lane w, and every word of L in scalars
  const uint64_t L = lane < words ? bits[(int64_t)lane * fstride + s] : 0ull;
  uint64_t Lw[kLaneWords];
#pragma unroll
  for (int w = 0; w < kLaneWords; w++) Lw[w] = w < words ? readlane_u64(L, w) : 0ull;

  // delta+(L) \ L and the boundary: lane l walks nodes 64 ww + l of L
  uint64_t acc[kLaneWords];
#pragma unroll
  for (int w = 0; w < kLaneWords; w++) acc[w] = 0;
  uint64_t bdw = 0;                                   // boundary word `lane`
  int64_t tl = 0, ml = 0, tb = 0, mb = 0;
#pragma unroll
  for (int ww = 0; ww < kLaneWords; ww++) {
    if (ww >= words) break;
    const int v = ww * 64 + lane;
    const bool in = (Lw[ww] >> lane) & 1ull;
    bool leaves = false;
#pragma unroll
    for (int w = 0; w < kLaneWords; w++) {
      if (w >= words) break;
      const uint64_t x = in ? succ[(int64_t)v * words + w] & ~Lw[w] : 0ull;
      acc[w] |= x;
      leaves |= x != 0;
    }
    const uint64_t bmask = __ballot(in && leaves);
    if (lane == ww) bdw = bmask;
    if (in) {
      const int32_t tv = T[v], mv = M[v];
      tl += tv;
      ml += mv;
      if (leaves) {
        tb += tv;
        mb += mv;
      }
    }
  }
  uint64_t out = 0;                                   // word `lane` of delta+(L) \ L
#pragma unroll
  for (int w = 0; w < kLaneWords; w++) {
    if (w >= words) break;
    const uint64_t r = wave_or_u64(acc[w]);
    if (lane == w) out = r;
  }
  // delta-(delta+(L) \ L) \ L, and M of both sets
#pragma unroll
  for (int w = 0; w < kLaneWords; w++) acc[w] = 0;
  int64_t ao = 0;
#pragma unroll
  for (int ww = 0; ww < kLaneWords; ww++) {
    if (ww >= words) break;
    const int v = ww * 64 + lane;
    const bool in = (readlane_u64(out, ww) >> lane) & 1ull;
    if (!in) continue;
    ao += M[v];
#pragma unroll
    for (int w = 0; w < kLaneWords; w++) {
      if (w >= words) break;
      acc[w] |= pred[(int64_t)v * words + w] & ~Lw[w];
    }
  }
  int64_t ai = 0;
#pragma unroll
  for (int w = 0; w < kLaneWords; w++) {
    if (w >= words) break;
    const uint64_t in2w = wave_or_u64(acc[w]);        // word w, the same on every lane
    if ((in2w >> lane) & 1ull) ai += M[w * 64 + lane];
  }
  tl = wave_sum_i64(tl);
  ml = wave_sum_i64(ml);
  tb = wave_sum_i64(tb);
  mb = wave_sum_i64(mb);
  ao = wave_sum_i64(ao);
  ai = wave_sum_i64(ai);
  const int sz = (int)wave_sum_i64(lane < words ? __popcll(L) : 0);
  if (lane < words) bd[(int64_t)lane * fstride + s] = bdw;
  if (lane == 0) {
    size[s] = sz;
    Tsum[s] = (int32_t)tl;
    Msum[s] = (int32_t)ml;
    Tbd[s] = (int32_t)tb;
    Mbd[s] = (int32_t)mb;
    A[s] = (int32_t)(ao + ai);
    w_out[s] = (int32_t)(tl - tb + 1);
  }
}

__global__ void k_row_widths(int64_t F, const int32_t* w, int64_t* padded) {
  const int64_t s = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (s < F) padded[s] = row_slot(w[s]);
}

// Rows are right-aligned inside their padded slots: row s ends on a
// kRowAlign boundary, so every column counted from the row end is made of
// whole 128-byte lines, and at least kGuard padding cells separate it from
// the previous row.
__global__ void k_row_align(int64_t F, const int32_t* w, int64_t* row_off) {
  const int64_t s = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
  if (s < F) row_off[s] += row_slot(w[s]) - w[s];
}

// ------------------------------------------------------------------ pairs

// Subset test of family members i and j (word-major storage).
__device__ __forceinline__ bool is_subset(const uint64_t* bits, int64_t fstride, int words,
                                          int64_t i, int64_t j) {
  for (int w = 0; w < words; w++)
    if (bits[(int64_t)w * fstride + i] & ~bits[(int64_t)w * fstride + j]) return false;
  return true;
}

// Predecessors of target j: i < j with L_i a proper subset of L_j.  The
// family is sorted by size, so every proper subset has a smaller index;
// equal sizes are never proper subsets.
__global__ __launch_bounds__(256) void k_pair_count(int64_t F, int words, int64_t fstride,
                                                    const uint64_t* bits, const int32_t* size,
                                                    int64_t* counts) {
  const int64_t j = blockIdx.x;
  __shared__ int64_t acc;
  if (threadIdx.x == 0) acc = 0;
  __syncthreads();
  int64_t c = 0;
  const int sj = size[j];
  for (int64_t i = threadIdx.x; i < j; i += blockDim.x)
    if (size[i] < sj && is_subset(bits, fstride, words, i, j)) c++;
  atomicAdd((unsigned long long*)&acc, (unsigned long long)c);
  __syncthreads();
  if (threadIdx.x == 0) counts[j] = acc;
}

// Pair data of (L = L_i, L' = L_j), in ascending i for every target j:
//   dt = T((L' \ L) \ bd(L')) = T(L' \ bd(L')) - T(L) + T(L & bd(L'))
//   dm = M(bd(L') \ L)        = M(bd(L')) - M(L & bd(L'))
//   c  = 2 M(L' \ L) + A(L')  = 2 (M(L') - M(L)) + A(L')
// so that the step of Algorithm 1 from (L, t, m) is admitted iff
// m + c <= B and then lands on (L', t + dt) with cache m + dm.  Only the
// two sums over L & bd(L') depend on the pair; bd(L') is small.
// walg[j] = sum over predecessors of w_i.
__global__ __launch_bounds__(256) void k_pair_write(
    int64_t F, int words, int64_t fstride, const uint64_t* bits, const uint64_t* bd,
    const int32_t* size, const int32_t* Tsum, const int32_t* Msum, const int32_t* Tbd,
    const int32_t* Mbd, const int32_t* A, const int32_t* w, const int32_t* T, const int32_t* M,
    const int64_t* pred_ptr, int32_t* pidx, int32_t* pdt, int32_t* pdm, int32_t* pc,
    int64_t* walg) {
  const int64_t j = blockIdx.x;
  __shared__ int64_t base;
  __shared__ int64_t wsum;
  __shared__ int32_t wave_cnt[4];
  if (threadIdx.x == 0) {
    base = pred_ptr[j];
    wsum = 0;
  }
  __syncthreads();
  const int sj = size[j];
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
  int64_t my_w = 0;
  for (int64_t i0 = 0; i0 < j; i0 += blockDim.x) {
    const int64_t i = i0 + threadIdx.x;
    const bool is = i < j && size[i] < sj && is_subset(bits, fstride, words, i, j);
    const uint64_t mask = __ballot(is);
    const int before = __popcll(mask & ((1ull << lane) - 1));
    if (lane == 0) wave_cnt[wv] = __popcll(mask);
    __syncthreads();
    int64_t off = base;
    for (int q = 0; q < wv; q++) off += wave_cnt[q];
    if (is) {
      int64_t ti = 0, mi = 0;
      for (int ww = 0; ww < words; ww++) {
        const uint64_t x = bits[(int64_t)ww * fstride + i] & bd[(int64_t)ww * fstride + j];
        ti += word_cost(x, ww, T);
        mi += word_cost(x, ww, M);
      }
      const int64_t p = off + before;
      pidx[p] = (int32_t)i;
      pdt[p] = (int32_t)((int64_t)Tsum[j] - Tbd[j] - Tsum[i] + ti);
      pdm[p] = (int32_t)((int64_t)Mbd[j] - mi);
      pc[p] = (int32_t)(2 * ((int64_t)Msum[j] - Msum[i]) + A[j]);
      my_w += w[i];
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int64_t tot = 0;
      for (int q = 0; q < (int)(blockDim.x / kWave); q++) tot += wave_cnt[q];
      base += tot;
    }
    __syncthreads();
  }
  atomicAdd((unsigned long long*)&wsum, (unsigned long long)my_w);
  __syncthreads();
  if (threadIdx.x == 0) walg[j] = wsum;
}

// ------------------------------------------------------------ scan / sum

// Exclusive scan of in[0..count) into out[0..count]; one workgroup.
__global__ __launch_bounds__(1024) void k_scan(const int64_t* in, int64_t* out, int64_t count) {
  __shared__ int64_t buf[1024];
  __shared__ int64_t carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  for (int64_t b = 0; b < count; b += 1024) {
    const int64_t i = b + threadIdx.x;
    const int64_t x = i < count ? in[i] : 0;
    buf[threadIdx.x] = x;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
      const int64_t y = threadIdx.x >= (unsigned)off ? buf[threadIdx.x - off] : 0;
      __syncthreads();
      buf[threadIdx.x] += y;
      __syncthreads();
    }
    if (i < count) out[i] = carry + buf[threadIdx.x] - x;
    __syncthreads();
    if (threadIdx.x == 1023) carry += buf[1023];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[count] = carry;
}

__global__ __launch_bounds__(1024) void k_sum(const int64_t* in, int64_t count, int64_t* out) {
  __shared__ int64_t acc;
  if (threadIdx.x == 0) acc = 0;
  __syncthreads();
  int64_t s = 0;
  for (int64_t i = threadIdx.x; i < count; i += blockDim.x) s += in[i];
  atomicAdd((unsigned long long*)&acc, (unsigned long long)s);
  __syncthreads();
  if (threadIdx.x == 0) *out = acc;
}

}  // namespace

// ============================================================== launchers

hipError_t launch_pack(const PackList& L, void* dst, hipStream_t s) {
  if (L.n <= 0) return hipSuccess;
  int64_t most = 0;
  for (int q = 0; q < L.n; q++) most = std::max<int64_t>(most, L.seg[q].bytes / 4);
  const unsigned gx = (unsigned)std::max<int64_t>(1, std::min<int64_t>((most + 255) / 256, 64));
  hipLaunchKernelGGL(k_pack, dim3(gx, (unsigned)L.n), dim3(256), 0, s, L,
                     static_cast<uint32_t*>(dst));
  return hipGetLastError();
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
  hipLaunchKernelGGL(k_zero_u64, dim3(1), dim3(256), 0, s, static_cast<uint64_t*>(p),
                     (int64_t)(bytes / 8));
  return hipGetLastError();
}

hipError_t launch_graph_masks(rc_graph g, const int32_t* d_row_ptr, const int32_t* d_col_idx,
                              hipStream_t s) {
  const int64_t cnt = (int64_t)g->n * g->words;
  hipLaunchKernelGGL(k_zero_u64, dim3(64), dim3(256), 0, s, g->dSucc, cnt);
  hipLaunchKernelGGL(k_zero_u64, dim3(64), dim3(256), 0, s, g->dPred, cnt);
  hipLaunchKernelGGL(k_graph_masks, dim3((g->n + 255) / 256), dim3(256), 0, s, g->n, g->words,
                     d_row_ptr, d_col_idx, g->dSucc, g->dPred);
  return hipGetLastError();
}

hipError_t launch_ancestors(rc_graph g, uint64_t* anc, hipStream_t s) {
  const size_t lds_closure = sizeof(uint64_t) * (size_t)g->n * g->words;
  if (g->words <= kClosureWords && (int64_t)g->n * g->words <= kClosureItems * kClosureThreads) {
    hipLaunchKernelGGL(k_ancestors_closure, dim3(1), dim3(kClosureThreads), lds_closure, s, g->n,
                       g->words, g->dPred, anc);
    return hipGetLastError();
  }
  const size_t lds_wave = sizeof(uint64_t) * (size_t)g->n * g->words +
                          sizeof(int32_t) * ((size_t)g->n + 1 + g->num_pred_edges + g->n);
  if (lds_wave <= 64 * 1024) {
    hipLaunchKernelGGL(k_ancestors_wave, dim3(1), dim3(kWave), lds_wave, s, g->n, g->words,
                       g->num_pred_edges, g->dByDepth, g->dPredPtr, g->dPredIdx, anc);
    return hipGetLastError();
  }
  const size_t lds = sizeof(uint64_t) * (size_t)g->n * g->words +
                     sizeof(int32_t) * ((size_t)g->n + 1 + g->num_pred_edges + g->n +
                                        g->num_depths + 1);
  if (lds <= 64 * 1024) {
    hipLaunchKernelGGL(k_ancestors<true>, dim3(1), dim3(1024), lds, s, g->n, g->words,
                       g->num_depths, g->num_pred_edges, g->dByDepth, g->dDepthPtr, g->dPredPtr,
                       g->dPredIdx, anc);
  } else {
    hipLaunchKernelGGL(k_ancestors<false>, dim3(1), dim3(1024), 0, s, g->n, g->words,
                       g->num_depths, g->num_pred_edges, g->dByDepth, g->dDepthPtr, g->dPredPtr,
                       g->dPredIdx, anc);
  }
  return hipGetLastError();
}

hipError_t launch_pruned_candidates(rc_graph g, const uint64_t* anc, uint64_t* cand,
                                    hipStream_t s) {
  hipLaunchKernelGGL(k_pruned_candidates, dim3(32), dim3(256), 0, s, g->n, g->words, anc, cand);
  return hipGetLastError();
}

hipError_t launch_enum_exact(rc_graph g, uint64_t* cand, int64_t cap, int32_t* lvl,
                             DevStatus* st, hipStream_t s) {
  hipLaunchKernelGGL(k_enum_start, dim3(1), dim3(64), 0, s, g->words, cand, lvl, st);
  for (int lev = 0; lev < g->n; lev++) {
    hipLaunchKernelGGL(k_enum_level, dim3(512), dim3(256), 0, s, g->n, g->words, lev, g->dSucc,
                       g->dPred, cand, cap, lvl, st);
    hipLaunchKernelGGL(k_enum_close, dim3(1), dim3(1), 0, s, lev, cap, lvl, st);
  }
  return hipGetLastError();
}

hipError_t launch_rank(rc_graph g, int32_t mode, const uint64_t* cand, int64_t ncand_max,
                       const int32_t* lvl, uint64_t* bits, int64_t fstride, DevStatus* st,
                       hipStream_t s) {
  if (mode == RC_FAMILY_PRUNED) {
    hipLaunchKernelGGL(k_rank_pruned, dim3(1), dim3(1024), 0, s, g->words, g->n, cand, bits,
                       fstride, st);
  } else {
    hipLaunchKernelGGL(k_rank, dim3((unsigned)((ncand_max + 255) / 256)), dim3(256), 0, s,
                       g->words, g->n, cand, lvl, bits, fstride, st);
  }
  return hipGetLastError();
}

hipError_t launch_set_quantities(rc_family f, hipStream_t s) {
  rc_graph g = f->g;
  const int per_block = 256 / kWave;
  const dim3 grid((unsigned)((f->F + per_block - 1) / per_block));
  const size_t lds = 2 * sizeof(uint64_t) * (size_t)g->n * g->words;
  if (g->words <= kLaneWords) {
    if (lds <= 64 * 1024)
      hipLaunchKernelGGL(k_set_quantities_lanes<true>, grid, dim3(256), lds, s, f->F, g->n,
                         g->words, f->fstride, f->bits, g->dSucc, g->dPred, g->dT, g->dM, f->bd,
                         f->size, f->Tsum, f->Msum, f->Tbd, f->Mbd, f->A, f->w);
    else
      hipLaunchKernelGGL(k_set_quantities_lanes<false>, grid, dim3(256), 0, s, f->F, g->n,
                         g->words, f->fstride, f->bits, g->dSucc, g->dPred, g->dT, g->dM, f->bd,
                         f->size, f->Tsum, f->Msum, f->Tbd, f->Mbd, f->A, f->w);
    return hipGetLastError();
  }
  if (lds <= 64 * 1024)
    hipLaunchKernelGGL(k_set_quantities<true>, grid, dim3(256), lds, s, f->F, g->n, g->words,
                       f->fstride, f->bits, g->dSucc, g->dPred, g->dT, g->dM, f->bd, f->size,
                       f->Tsum, f->Msum, f->Tbd, f->Mbd, f->A, f->w);
  else
    hipLaunchKernelGGL(k_set_quantities<false>, grid, dim3(256), 0, s, f->F, g->n, g->words,
                       f->fstride, f->bits, g->dSucc, g->dPred, g->dT, g->dM, f->bd, f->size,
                       f->Tsum, f->Msum, f->Tbd, f->Mbd, f->A, f->w);
  return hipGetLastError();
}

hipError_t launch_row_widths(rc_family f, int64_t* padded, hipStream_t s) {
  hipLaunchKernelGGL(k_row_widths, dim3((unsigned)((f->F + 255) / 256)), dim3(256), 0, s, f->F,
                     f->w, padded);
  return hipGetLastError();
}

hipError_t launch_row_align(rc_family f, hipStream_t s) {
  hipLaunchKernelGGL(k_row_align, dim3((unsigned)((f->F + 255) / 256)), dim3(256), 0, s, f->F,
                     f->w, f->row_off);
  return hipGetLastError();
}

hipError_t launch_pair_count(rc_family f, int64_t* counts, hipStream_t s) {
  hipLaunchKernelGGL(k_pair_count, dim3((unsigned)f->F), dim3(256), 0, s, f->F, f->g->words,
                     f->fstride, f->bits, f->size, counts);
  return hipGetLastError();
}

hipError_t launch_scan(const int64_t* in, int64_t* out, int64_t count, int64_t, hipStream_t s) {
  hipLaunchKernelGGL(k_scan, dim3(1), dim3(1024), 0, s, in, out, count);
  return hipGetLastError();
}

hipError_t launch_pair_write(rc_family f, int64_t* walg_per_target, hipStream_t s) {
  rc_graph g = f->g;
  hipLaunchKernelGGL(k_pair_write, dim3((unsigned)f->F), dim3(256), 0, s, f->F, g->words,
                     f->fstride, f->bits, f->bd, f->size, f->Tsum, f->Msum, f->Tbd, f->Mbd, f->A,
                     f->w, g->dT, g->dM, f->pred_ptr, f->pidx, f->pdt, f->pdm, f->pc,
                     walg_per_target);
  return hipGetLastError();
}

hipError_t launch_sum(const int64_t* in, int64_t count, int64_t* out, hipStream_t s) {
  hipLaunchKernelGGL(k_sum, dim3(1), dim3(1024), 0, s, in, count, out);
  return hipGetLastError();
}

}  // namespace rcdp
