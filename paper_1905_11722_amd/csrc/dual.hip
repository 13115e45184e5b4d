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
// Layout: D[L * W + m], uint32, kDualNone where no chain reaches (L, m).
// One launch per group of equal-size sets (sets of equal size never contain
// each other), a thread per target cell looping over the target's pairs
// (the family's predecessor lists, read through wave-uniform scalar loads).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "rc_internal.h"

namespace rcdp {

namespace {

constexpr int kDualThreads = 256;
constexpr uint32_t kDualNone = 0xFFFFFFFFu;

__global__ void k_dual_init(uint32_t* D, int64_t cells, DevStatus* st) {
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < cells;
       x += (int64_t)gridDim.x * blockDim.x)
    D[x] = x == 0 ? 0u : kDualNone;                 // (empty set, m = 0): t = 0
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    st->error = 0;
    st->t_sel = -1;
    st->m_sel = -1;
  }
}

// Block (x, y): cells [x * kDualThreads, (x + 1) * kDualThreads) of target
// lb + y.
template <bool kTC>
__global__ __launch_bounds__(kDualThreads) void k_dual_level(
    int64_t lb, int32_t W, int32_t B, const int64_t* __restrict__ pred_ptr,
    const int32_t* __restrict__ pidx, const int32_t* __restrict__ pdt,
    const int32_t* __restrict__ pdm, const int32_t* __restrict__ pc, uint32_t* __restrict__ D) {
  const int64_t j = lb + blockIdx.y;
  const int32_t mp = blockIdx.x * kDualThreads + threadIdx.x;
  if (mp >= W) return;
  uint32_t acc = kDualNone;
  const int64_t p0 = pred_ptr[j], p1 = pred_ptr[j + 1];
  for (int64_t p = p0; p < p1; ++p) {
    const int32_t m = mp - pdm[p];                 // source cell: memory before the step
    if (m < 0 || m > B - pc[p]) continue;          // budget test of Algorithm 1: m + c <= B
    const uint32_t x = D[(int64_t)pidx[p] * W + m];
    if (x == kDualNone) continue;
    const uint32_t y = x + (uint32_t)pdt[p];
    if (kTC)
      acc = min(acc, y);                           // kDualNone is the largest value
    else
      acc = acc == kDualNone ? y : max(acc, y);
  }
  D[j * (int64_t)W + mp] = acc;
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
    if (x == kDualNone) continue;
    best = tc ? min(best, (unsigned long long)x) : max(best, (unsigned long long)x + 1);
  }
  if (tc)
    atomicMin(&s_best, best);
  else
    atomicMax(&s_best, best);
  __syncthreads();
  const bool found = tc ? s_best != kDualNone : s_best != 0;
  if (found) {
    const uint32_t t = (uint32_t)(tc ? s_best : s_best - 1);
    for (int32_t m = threadIdx.x; m < W; m += blockDim.x)
      if (row[m] == t) {
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

hipError_t launch_dual(rc_family f, int32_t B, int32_t W, int objective, uint32_t* D,
                       DevStatus* st, hipEvent_t e0, hipEvent_t e1, hipStream_t s) {
  const int64_t cells = f->F * (int64_t)W;
  const unsigned grid0 = (unsigned)std::min<int64_t>((cells + 255) / 256, 4096);
  hipLaunchKernelGGL(k_dual_init, dim3(grid0), dim3(256), 0, s, D, cells, st);
  if (e0 && hipEventRecord(e0, s) != hipSuccess) return hipErrorUnknown;
  const bool tc = objective == RC_TIME_CENTRIC;
  const unsigned tiles = (unsigned)((W + kDualThreads - 1) / kDualThreads);
  const int64_t L = (int64_t)f->level_ptr.size() - 1;
  for (int64_t l = 0; l < L; l++) {
    const int64_t lb = std::max<int64_t>(f->level_ptr[l], 1), le = f->level_ptr[l + 1];
    if (le <= lb) continue;
    if (tc)
      hipLaunchKernelGGL(k_dual_level<true>, dim3(tiles, (unsigned)(le - lb)), dim3(kDualThreads),
                         0, s, lb, W, B, f->pred_ptr, f->pidx, f->pdt, f->pdm, f->pc, D);
    else
      hipLaunchKernelGGL(k_dual_level<false>, dim3(tiles, (unsigned)(le - lb)),
                         dim3(kDualThreads), 0, s, lb, W, B, f->pred_ptr, f->pidx, f->pdt, f->pdm,
                         f->pc, D);
  }
  if (e1 && hipEventRecord(e1, s) != hipSuccess) return hipErrorUnknown;
  hipLaunchKernelGGL(k_dual_select, dim3(1), dim3(kDualThreads), 0, s,
                     D + (f->F - 1) * (int64_t)W, W, tc ? 1 : 0, st);
  return hipGetLastError();
}

}  // namespace rcdp
