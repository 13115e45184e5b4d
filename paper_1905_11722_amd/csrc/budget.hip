// The smallest feasible budget of a family, on the device.
//
// The experiments of Section 5 run at the smallest budget B for which the
// General Recomputation Problem has a solution, found by binary search.
// Whether B admits a solution does not depend on t: every row minimum of the
// table of Algorithm 1 equals f[L], the same recursion with the t axis taken
// out,
//     f[empty] = 0,   f[L'] = min over L < L' in the family of f[L] + dm(L, L')
//                     over the pairs with f[L] + c(L, L') <= B,
// and B is feasible exactly when f[V] is finite.  Feasibility is monotone
// in B and B = 2 M(V) is always feasible (the one-segment chain {V} peaks at
// 2 M(V)), so the search runs over [0, 2 M(V)].  Each round evaluates 64
// budgets at once, one per lane, spread over the open interval between the
// largest budget known infeasible and the smallest known feasible; each
// round shrinks that interval 65-fold, so at most three rounds reach a
// budget range of 2^16.  When f fits LDS, 16 waves share a target's pairs
// (k_min_budget_waves); otherwise one wave walks them with f in global
// scratch (k_min_budget).
#include <hip/hip_runtime.h>

#include "rc_internal.h"

namespace rcdp {

namespace {

constexpr int kLanes = 64;

typedef const __attribute__((address_space(4))) int32_t cint32;
typedef const __attribute__((address_space(4))) int64_t cint64;

// f of every set for the 64 budgets of a round: [F][64], in LDS when it
// fits, else in global scratch.  One wave, so a lane reads back what it
// wrote in program order.
template <typename FT, bool kLds>
__global__ __launch_bounds__(kLanes) void k_min_budget(int64_t F, int32_t hi0,
                                                       const int64_t* pred_ptr,
                                                       const int32_t* pidx, const int32_t* pdm,
                                                       const int32_t* pc, FT* fglob,
                                                       DevStatus* st) {
  constexpr FT kInfF = (FT)~(FT)0;                 // every finite f is below it
  extern __shared__ __attribute__((aligned(16))) unsigned char flds_raw[];
  FT* f = kLds ? reinterpret_cast<FT*>(flds_raw) : fglob;
  const int lane = threadIdx.x;
  cint64* pp = (cint64*)pred_ptr;
  cint32* pi = (cint32*)pidx;
  cint32* pm = (cint32*)pdm;
  cint32* pcc = (cint32*)pc;
  int32_t lo = -1, hi = hi0;                       // lo infeasible, hi feasible
  while (hi - lo > 1) {
    const int64_t span = hi - lo;
    const int32_t B = lo + (int32_t)(((int64_t)(lane + 1) * span + kLanes) / (kLanes + 1));
    f[lane] = 0;                                   // the empty set
    for (int64_t j = 1; j < F; j++) {
      FT best = kInfF;
      const int64_t p0 = pp[j], p1 = pp[j + 1];
      for (int64_t p = p0; p < p1; p++) {
        const int32_t i = pi[p];
        const FT fi = f[i * kLanes + lane];
        if (fi != kInfF && (int64_t)fi + pcc[p] <= B) {
          const FT cand = (FT)(fi + pm[p]);
          best = cand < best ? cand : best;
        }
      }
      f[j * kLanes + lane] = best;
      if (!kLds) __threadfence_block();
    }
    const bool ok = f[(F - 1) * kLanes + lane] != kInfF;
    const unsigned long long bal = __ballot(ok);
    // the lane of budget hi0 or of a budget above the last feasible one is
    // feasible; the smallest feasible lane bounds the new interval
    const int first = bal ? __ffsll((long long)bal) - 1 : kLanes;
    const int32_t Bfirst = __shfl(B, first < kLanes ? first : 0, kLanes);
    const int32_t Bprev = __shfl(B, first > 0 ? first - 1 : 0, kLanes);
    if (first < kLanes) hi = Bfirst;
    if (first > 0) lo = first < kLanes ? Bprev : __shfl(B, kLanes - 1, kLanes);
    __syncthreads();
  }
  if (lane == 0) st->bmin = hi;
}

// The same search with the pairs of a target spread over kMbWaves waves:
// wave w, lane q holds pair p0 + kMbWaves q + w of the target (one coalesced
// load per wave, issued a target ahead), every wave relaxes its pairs for
// the 64 budgets (lane = budget, pair values taken with readlane), and the
// waves' partial minima meet in LDS.  Two barriers per target instead of a
// dependent scalar load per pair.
constexpr int kMbWaves = 16;
constexpr int kMbChunk = kMbWaves * kLanes;          // pairs per target and pass

template <typename FT>
__global__ __launch_bounds__(kMbChunk) void k_min_budget_waves(int64_t F, int32_t hi0,
                                                                const int64_t* pred_ptr,
                                                                const int32_t* pidx,
                                                                const int32_t* pdm,
                                                                const int32_t* pc,
                                                                DevStatus* st) {
  constexpr FT kInfF = (FT)~(FT)0;
  extern __shared__ __attribute__((aligned(16))) unsigned char flds_raw[];
  FT* f = reinterpret_cast<FT*>(flds_raw);               // [F][64]
  __shared__ uint32_t red[kMbWaves][kLanes];
  const int lane = threadIdx.x & (kLanes - 1);
  const int wave = threadIdx.x / kLanes;
  cint64* pp = (cint64*)pred_ptr;
  // pair p0 + kMbWaves * lane + wave of target j (j < F), chunk base p0
  auto load = [&](int64_t j, int64_t base, int32_t& i, int32_t& dm, int32_t& c) {
    i = -1;
    dm = 0;
    c = 0;
    if (j >= F) return;
    const int64_t p = base + (int64_t)kMbWaves * lane + wave;
    if (p < pp[j + 1]) {
      i = pidx[p];
      dm = pdm[p];
      c = pc[p];
    }
  };
  int32_t lo = -1, hi = hi0;                           // lo infeasible, hi feasible
  while (hi - lo > 1) {
    const int64_t span = hi - lo;
    const int32_t B = lo + (int32_t)(((int64_t)(lane + 1) * span + kLanes) / (kLanes + 1));
    if (wave == 0) f[lane] = 0;                        // the empty set
    int32_t ni, ndm, nc;                               // the next target's first chunk
    load(1, F > 1 ? pp[1] : 0, ni, ndm, nc);
    __syncthreads();
    for (int64_t j = 1; j < F; j++) {
      const int64_t p0 = pp[j], p1 = pp[j + 1];
      int32_t ci = ni, cdm = ndm, cc = nc;
      load(j + 1, j + 1 < F ? pp[j + 1] : 0, ni, ndm, nc);
      uint32_t best = kInfF;
      for (int64_t base = p0; base < p1; base += kMbChunk) {
        if (base != p0) load(j, base, ci, cdm, cc);
        // pairs of this wave in the chunk: base + kMbWaves * q + wave < p1
        const int64_t rem = p1 - base - wave;
        const int nq = rem <= 0 ? 0 : (int)min<int64_t>(kLanes, (rem + kMbWaves - 1) / kMbWaves);
        for (int q = 0; q < nq; q++) {
          const int32_t i = __builtin_amdgcn_readlane(ci, q);
          const int32_t dm = __builtin_amdgcn_readlane(cdm, q);
          const int32_t c = __builtin_amdgcn_readlane(cc, q);
          const uint32_t fi = f[(int64_t)i * kLanes + lane];
          if (fi != kInfF && (int64_t)fi + c <= B) {
            const uint32_t cand = fi + (uint32_t)dm;
            best = cand < best ? cand : best;
          }
        }
      }
      red[wave][lane] = best;
      __syncthreads();
      if (wave == 0) {
        uint32_t m = red[0][lane];
#pragma unroll
        for (int w = 1; w < kMbWaves; w++) m = min(m, red[w][lane]);
        f[j * kLanes + lane] = (FT)m;
      }
      __syncthreads();
    }
    const bool ok = f[(F - 1) * kLanes + lane] != kInfF;
    const unsigned long long bal = __ballot(ok);
    const int first = bal ? __ffsll((long long)bal) - 1 : kLanes;
    const int32_t Bfirst = __shfl(B, first < kLanes ? first : 0, kLanes);
    const int32_t Bprev = __shfl(B, first > 0 ? first - 1 : 0, kLanes);
    if (first < kLanes) hi = Bfirst;
    if (first > 0) lo = first < kLanes ? Bprev : __shfl(B, kLanes - 1, kLanes);
    __syncthreads();
  }
  if (threadIdx.x == 0) st->bmin = hi;
}

}  // namespace

// Value type and home of f: 16 bits when every finite value (at most
// 2 M(V)) fits below the infinity code, LDS when [F][64] fits in 64 KB.
static int min_budget_kind(rc_family f, int32_t hi0) {
  // the multi-wave kernel keeps 4 KB of partial minima in LDS beside f
  if (hi0 < 0xFFFF && (size_t)f->F * kLanes * 2 <= 60 * 1024) return 0;
  if ((size_t)f->F * kLanes * 4 <= 60 * 1024) return 1;
  return 2;
}

size_t min_budget_scratch_bytes(rc_family f, int32_t hi0) {
  return min_budget_kind(f, hi0) == 2 ? sizeof(uint32_t) * (size_t)f->F * kLanes : 0;
}

hipError_t launch_min_budget(rc_family f, int32_t hi0, uint32_t* scratch, hipStream_t s) {
  const int kind = min_budget_kind(f, hi0);
  if (kind == 0) {
    hipLaunchKernelGGL((k_min_budget_waves<uint16_t>), dim3(1), dim3(kMbChunk),
                       sizeof(uint16_t) * (size_t)f->F * kLanes, s, f->F, hi0, f->pred_ptr,
                       f->pidx, f->pdm, f->pc, f->status);
    return hipGetLastError();
  }
  if (kind == 1) {
    hipLaunchKernelGGL((k_min_budget_waves<uint32_t>), dim3(1), dim3(kMbChunk),
                       sizeof(uint32_t) * (size_t)f->F * kLanes, s, f->F, hi0, f->pred_ptr,
                       f->pidx, f->pdm, f->pc, f->status);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((k_min_budget<uint32_t, false>), dim3(1), dim3(kLanes), 0, s, f->F, hi0,
                     f->pred_ptr, f->pidx, f->pdm, f->pc, scratch, f->status);
  return hipGetLastError();
}

}  // namespace rcdp
