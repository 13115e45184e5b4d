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

}  // namespace

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
