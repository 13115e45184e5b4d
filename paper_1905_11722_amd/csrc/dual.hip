// Memory-indexed form of Algorithm 1's recursion (Section 4.2, Appendix A).
//
// Algorithm 1 walks states (L, t, m) -- a chain ending at lower set L with
// forward time t and cached memory m -- and keeps, per (L, t), the least m.
// A pair L < L' moves (L, t, m) to (L', t + dt, m + dm) when m + c <= B; the
// test depends on m alone.  This table keeps, per (L, m), the least t (time
// centric) or the greatest t (memory centric, Section 4.4) instead: a later
// step adds the same time to two states of equal memory, so the kept one is
// never worse, and the optimum over row V is Algorithm 1's t* with
// opt[V, t*] = the least m that attains it.  Rows span m in [0, W),
// W = min(B, M(V)) + 1 (every cached memory is M(U) for a node set U), so the
// budget test becomes a window on the source index: target cell m' reads
// source cell m' - dm when 0 <= m' - dm <= B - c.
//
// Layout: D[L * W + m], uint32.  Time centric: t, kDualNone (the largest
// value) where no chain reaches (L, m); memory centric: t + 1, 0 where none
// does, so that both combine with one atomic min / max.
// One launch per group of equal-size sets (sets of equal size never contain
// each other).  Block (x, y, z): 256 cells of target y of the group and the
// z-th run of kDualPairs of its pairs (read through wave-uniform scalar
// loads); a thread issues the source loads of kDualBatch pairs together and
// folds its candidate into the target cell with one atomic.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <vector>

#include "rc_internal.h"
#include "dual.h"
#include "schedule.h"

namespace rcdp {

namespace {

constexpr int kDualThreads = 256;
constexpr int kDualPairs = 4;                       // pairs per block
constexpr int kDualBatch = 4;                       // source loads in flight per thread
constexpr uint32_t kDualNone = 0xFFFFFFFFu;

__global__ void k_dual_init(uint32_t* D, int64_t cells, int tc, DevStatus* st) {
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < cells;
       x += (int64_t)gridDim.x * blockDim.x)
    D[x] = x == 0 ? (tc ? 0u : 1u) : (tc ? kDualNone : 0u);   // (empty set, m = 0): t = 0
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    st->error = 0;
    st->t_sel = -1;
    st->m_sel = -1;
  }
}

template <bool kTC>
__global__ __launch_bounds__(kDualThreads) void k_dual_level(
    int64_t lb, int32_t W, int32_t B, const int64_t* __restrict__ pred_ptr,
    const int32_t* __restrict__ pidx, const int32_t* __restrict__ pdt,
    const int32_t* __restrict__ pdm, const int32_t* __restrict__ pc, uint32_t* __restrict__ D) {
  constexpr uint32_t kNone = kTC ? kDualNone : 0u;
  const int64_t j = lb + blockIdx.y;
  const int32_t mp = blockIdx.x * kDualThreads + threadIdx.x;
  const int64_t q0 = pred_ptr[j], q1 = pred_ptr[j + 1];
  const int64_t p0 = q0 + (int64_t)blockIdx.z * kDualPairs;
  const int64_t p1 = min(q1, p0 + kDualPairs);
  if (mp >= W || p0 >= p1) return;
  uint32_t acc = kNone;
  for (int64_t pb = p0; pb < p1; pb += kDualBatch) {
    uint32_t x[kDualBatch];
    int32_t dt[kDualBatch];
#pragma unroll
    for (int k = 0; k < kDualBatch; k++) {
      // every load is issued (a pair past the run re-reads the run's first
      // one, a cell outside the window reads cell 0) and tested afterwards
      const int64_t p = pb + k < p1 ? pb + k : p0;
      const int32_t m = mp - pdm[p];                 // source cell: memory before the step
      const bool ok = pb + k < p1 && m >= 0 && m <= B - pc[p];   // m + c <= B (Algorithm 1)
      const uint32_t v = D[(int64_t)pidx[p] * W + (ok ? m : 0)];
      x[k] = ok ? v : kNone;
      dt[k] = pdt[p];
    }
#pragma unroll
    for (int k = 0; k < kDualBatch; k++) {
      if (x[k] == kNone) continue;
      const uint32_t y = x[k] + (uint32_t)dt[k];
      acc = kTC ? min(acc, y) : max(acc, y);
    }
  }
  if (acc == kNone) return;
  if (kTC)
    atomicMin(&D[j * (int64_t)W + mp], acc);
  else
    atomicMax(&D[j * (int64_t)W + mp], acc);
}

// t of the objective over row V and the least m that attains it.
__global__ __launch_bounds__(kDualThreads) void k_dual_select(const uint32_t* __restrict__ row,
                                                              int32_t W, int tc, DevStatus* st) {
  __shared__ unsigned long long s_best;             // TC: t; MC: t + 1 (0: none)
  __shared__ int32_t s_m;
  if (threadIdx.x == 0) {
    s_best = tc ? (unsigned long long)kDualNone : 0ull;
    s_m = INT32_MAX;
  }
  __syncthreads();
  unsigned long long best = tc ? (unsigned long long)kDualNone : 0ull;
  for (int32_t m = threadIdx.x; m < W; m += blockDim.x) {
    const uint32_t x = row[m];
    if (tc ? x == kDualNone : x == 0u) continue;
    best = tc ? min(best, (unsigned long long)x) : max(best, (unsigned long long)x);
  }
  if (tc)
    atomicMin(&s_best, best);
  else
    atomicMax(&s_best, best);
  __syncthreads();
  const bool found = tc ? s_best != kDualNone : s_best != 0;
  if (found) {
    const uint32_t code = (uint32_t)s_best;
    for (int32_t m = threadIdx.x; m < W; m += blockDim.x)
      if (row[m] == code) {
        atomicMin(&s_m, m);
        break;
      }
  }
  __syncthreads();
  if (threadIdx.x == 0 && found) {
    st->t_sel = (int32_t)(tc ? s_best : s_best - 1);
    st->m_sel = s_m;
  }
}

// Traceback through the table (Section 4.2's, read on cells (L, m)): from
// (V, m*, t*), the next set is the smallest family index L among the pairs
// L < L' whose cell (L, m - dm) passes the budget test and holds t - dt (one
// always does along an optimal chain: its state there is reachable, and a
// better one would give a better optimum).  The walk must end at (empty set,
// 0, 0); then the chain's strategy is evaluated (finish_schedule).  The
// pairs of a step are scanned kDualTraceThreads at a time; the first hit in
// family order is the lowest hitting thread of the first chunk with one.
constexpr int kDualTraceThreads = 512;

template <bool kTC>
__global__ __launch_bounds__(kDualTraceThreads) void k_dual_trace(
    int64_t F, int n, int words, int64_t fstride, const uint64_t* __restrict__ bits,
    const uint64_t* __restrict__ bd, const int32_t* __restrict__ A, const int32_t* __restrict__ T,
    const int32_t* __restrict__ M, const int64_t* __restrict__ pred_ptr,
    const int32_t* __restrict__ pidx, const int32_t* __restrict__ pdt,
    const int32_t* __restrict__ pdm, const int32_t* __restrict__ pc, int32_t B, int32_t W,
    const uint32_t* __restrict__ D, int64_t T_total, DevStatus* st, int32_t* chain, int32_t* seg,
    uint8_t* cached) {
  constexpr int kWaves = kDualTraceThreads / 64;
  __shared__ int32_t s_first[2][kWaves];
  __shared__ int32_t s_src[2][kDualTraceThreads];
  __shared__ int32_t s_dt[2][kDualTraceThreads];
  __shared__ int32_t s_dm[2][kDualTraceThreads];
  __shared__ int32_t s_chain[kMaxNodes + 1];
  __shared__ int32_t s_M[kMaxNodes];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid / 64;
  int64_t j = F - 1;
  int64_t t = st->t_sel, m = st->m_sel;
  int32_t k = 0;
  bool bad = t < 0 || m < 0 || m >= W;
  int par = 0;
  while (j != 0 && !bad) {
    if (k >= F || k > n) {                          // each step removes a node
      bad = true;
      break;
    }
    const int64_t p0 = pred_ptr[j], p1 = pred_ptr[j + 1];
    int32_t next_i = -1, next_dt = 0, next_dm = 0;
    for (int64_t base = p0; base < p1 && next_i < 0; base += kDualTraceThreads) {
      const int64_t p = base + tid;
      const bool valid = p < p1;
      const int64_t pq = valid ? p : p0;
      const int32_t i = pidx[pq], dt = pdt[pq], dm = pdm[pq], c = pc[pq];
      const int64_t ms = m - dm;                     // memory before the step
      const bool ok = valid && ms >= 0 && ms <= B - c;
      const uint32_t x = D[(int64_t)i * W + (ok ? ms : 0)];
      const bool reached = kTC ? x != kDualNone : x != 0u;
      const int64_t tx = kTC ? (int64_t)x : (int64_t)x - 1;
      const bool hit = ok && reached && tx + dt == t;
      const unsigned long long bal = __ballot(hit);
      if (lane == 0) s_first[par][wave] = bal ? wave * 64 + __ffsll((long long)bal) - 1 : INT32_MAX;
      s_src[par][tid] = i;
      s_dt[par][tid] = dt;
      s_dm[par][tid] = dm;
      __syncthreads();
      int32_t f = INT32_MAX;
#pragma unroll
      for (int q = 0; q < kWaves; q++) f = min(f, s_first[par][q]);
      if (f != INT32_MAX) {
        next_i = s_src[par][f];
        next_dt = s_dt[par][f];
        next_dm = s_dm[par][f];
      }
      par ^= 1;
    }
    if (next_i < 0) {
      bad = true;
      break;
    }
    if (tid == 0) chain[k] = (int32_t)j;
    k++;
    t -= next_dt;
    m -= next_dm;
    j = next_i;
  }
  if (t != 0 || m != 0) bad = true;                  // the walk must end at (empty set, 0, 0)
  __syncthreads();
  if (bad) {
    if (tid == 0) {
      st->error = 2;
      st->k = -1;
    }
    return;
  }
  finish_schedule<kDualTraceThreads>(k, n, words, fstride, bits, bd, A, T, M, T_total, st, chain,
                                     seg, cached, s_chain, s_M);
}

}  // namespace

hipError_t launch_dual_trace(rc_family f, int32_t B, int32_t W, int objective, const uint32_t* D,
                             DevStatus* st, int32_t* chain, int32_t* seg, uint8_t* cached,
                             hipStream_t s) {
  rc_graph g = f->g;
  if (objective == RC_TIME_CENTRIC)
    hipLaunchKernelGGL(k_dual_trace<true>, dim3(1), dim3(kDualTraceThreads), 0, s, f->F, g->n,
                       g->words, f->fstride, f->bits, f->bd, f->A, g->dT, g->dM, f->pred_ptr,
                       f->pidx, f->pdt, f->pdm, f->pc, B, W, D, g->T_total, st, chain, seg,
                       cached);
  else
    hipLaunchKernelGGL(k_dual_trace<false>, dim3(1), dim3(kDualTraceThreads), 0, s, f->F, g->n,
                       g->words, f->fstride, f->bits, f->bd, f->A, g->dT, g->dM, f->pred_ptr,
                       f->pidx, f->pdt, f->pdm, f->pc, B, W, D, g->T_total, st, chain, seg,
                       cached);
  return hipGetLastError();
}

hipError_t launch_dual(rc_family f, const std::vector<int64_t>& level_pairs, int32_t B, int32_t W,
                       int objective, uint32_t* D, DevStatus* st, hipEvent_t e0, hipEvent_t e1,
                       hipStream_t s) {
  const int64_t cells = f->F * (int64_t)W;
  const unsigned grid0 = (unsigned)std::min<int64_t>((cells + 255) / 256, 4096);
  const bool tc = objective == RC_TIME_CENTRIC;
  hipLaunchKernelGGL(k_dual_init, dim3(grid0), dim3(256), 0, s, D, cells, tc ? 1 : 0, st);
  if (e0 && hipEventRecord(e0, s) != hipSuccess) return hipErrorUnknown;
  const unsigned tiles = (unsigned)((W + kDualThreads - 1) / kDualThreads);
  const int64_t L = (int64_t)f->level_ptr.size() - 1;
  for (int64_t l = 0; l < L; l++) {
    const int64_t lb = std::max<int64_t>(f->level_ptr[l], 1), le = f->level_ptr[l + 1];
    if (le <= lb) continue;
    const dim3 grid(tiles, (unsigned)(le - lb),
                    (unsigned)((level_pairs[l] + kDualPairs - 1) / kDualPairs));
    if (grid.z == 0) continue;
    if (tc)
      hipLaunchKernelGGL(k_dual_level<true>, grid, dim3(kDualThreads), 0, s, lb, W, B,
                         f->pred_ptr, f->pidx, f->pdt, f->pdm, f->pc, D);
    else
      hipLaunchKernelGGL(k_dual_level<false>, grid, dim3(kDualThreads), 0, s, lb, W, B,
                         f->pred_ptr, f->pidx, f->pdt, f->pdm, f->pc, D);
  }
  if (e1 && hipEventRecord(e1, s) != hipSuccess) return hipErrorUnknown;
  hipLaunchKernelGGL(k_dual_select, dim3(1), dim3(kDualThreads), 0, s,
                     D + (f->F - 1) * (int64_t)W, W, tc ? 1 : 0, st);
  return hipGetLastError();
}

}  // namespace rcdp
