// The canonical strategy of a traced chain (Section 3), evaluated on the
// device from its definitions: V_i = L_i \ L_{i-1}, U_i = U_{i-1} plus the
// boundary of L_i, segment i needs M(U_{i-1}) + 2 M(V_i) + A(L_i) (Eq. 2,
// A(L) = M(delta+(L) \ L) + M(delta-(delta+(L)) \ L)), and the overhead is
// T(V \ U_k) (Eq. 1).  Shared by the traceback of the time-indexed table
// (fill.hip) and of the memory-indexed one (dual.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rc_internal.h"

namespace rcdp {
namespace sched {

constexpr int kWave = 64;

template <class V>
__device__ __forceinline__ V wave_sum(V x) {
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, kWave);
  return x;
}

template <class V>
__device__ __forceinline__ V wave_max(V x) {
  for (int off = 32; off > 0; off >>= 1) {
    const V y = __shfl_xor(x, off, kWave);
    x = y > x ? y : x;
  }
  return x;
}

}  // namespace sched

// Every thread of the block calls it after the walk: chain[0 .. k) holds the
// chain from V back to its first set; it is written back in increasing order
// (L_1 .. L_k), seg[n] (segment index of each node), cached[n] (1 iff in U_k)
// and st->{k, overhead, peak, cache_mem} are filled.  s_chain[k] and s_M[n]
// are LDS scratch of the caller.
//
// The chain's steps are evaluated together rather than one after another:
// a node v lies in V_i for exactly one i (the chain is increasing and ends
// at V), and it belongs to U_{i-1} exactly when some L_j with j < i has it
// in its boundary.  So with seg(v) = that i and first(v) = the least j whose
// boundary holds v, M(V_i) sums M_v over seg(v) = i, M(U_{i-1}) sums M_v
// over first(v) < i (a prefix over the steps), and U_k holds the nodes with
// a first(v).  Sums of memory stay below 2^31 (the graph's M(V) < 2^29);
// the segment sums and T(U_k) are carried in 64 bits.
template <int kThreads>
__device__ __forceinline__ void finish_schedule(int32_t k, int n, int words, int64_t fstride,
                                const uint64_t* __restrict__ bits, const uint64_t* __restrict__ bd,
                                const int32_t* __restrict__ A, const int32_t* __restrict__ T,
                                const int32_t* __restrict__ M, int64_t T_total, DevStatus* st,
                                int32_t* chain, int32_t* seg, uint8_t* cached, int32_t* s_chain,
                                int32_t* s_M) {
  using sched::kWave;
  constexpr int kWaves = kThreads / kWave;
  __shared__ int32_t s_seg[kMaxNodes];       // seg(v), -1 before it is known
  __shared__ int32_t s_first[kMaxNodes];     // first(v), INT32_MAX for a node never in a boundary
  __shared__ int32_t s_mv[kMaxNodes + 1];    // M(V_i)
  __shared__ int32_t s_gain[kMaxNodes + 1];  // M of the nodes U gains at step i
  __shared__ int64_t s_red[3][kWaves];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  for (int c = tid; c < k; c += kThreads) {
    s_chain[c] = chain[k - 1 - c];
    s_mv[c] = 0;
    s_gain[c] = 0;
  }
  for (int v = tid; v < n; v += kThreads) {
    s_seg[v] = -1;
    s_first[v] = INT32_MAX;
    s_M[v] = M[v];
  }
  __syncthreads();
  for (int c = tid; c < k; c += kThreads) chain[c] = s_chain[c];
  // one (step, word) per item: the nodes V_i of the step and the boundary of L_i
  for (int x = tid; x < k * words; x += kThreads) {
    const int c = x / words, wd = x - c * words;
    const int64_t base = (int64_t)wd * fstride;
    const uint64_t Li = bits[base + s_chain[c]];
    const uint64_t Lp = c > 0 ? bits[base + s_chain[c - 1]] : 0ull;
    uint64_t Bi = bd[base + s_chain[c]];
    int32_t mv = 0;
    for (uint64_t b = Li & ~Lp; b; b &= b - 1) {
      const int v = wd * 64 + __builtin_ctzll(b);
      s_seg[v] = c;
      mv += s_M[v];
    }
    if (mv) atomicAdd(&s_mv[c], mv);
    for (; Bi; Bi &= Bi - 1) atomicMin(&s_first[wd * 64 + __builtin_ctzll(Bi)], c);
  }
  __syncthreads();
  // per node: its segment, whether U_k holds it, and the step at which U gains it
  int64_t tu = 0;
  for (int v = tid; v < n; v += kThreads) {
    seg[v] = s_seg[v];
    const int32_t f = s_first[v];
    cached[v] = f < k ? 1 : 0;
    if (f < k) {
      atomicAdd(&s_gain[f], s_M[v]);
      tu += T[v];
    }
  }
  __syncthreads();
  // M(U_{i-1}): exclusive prefix of the gains, each thread a run of steps
  const int per = (k + kThreads - 1) / kThreads;
  const int c0 = min(k, tid * per), c1 = min(k, c0 + per);
  int64_t run = 0;
  for (int c = c0; c < c1; c++) run += s_gain[c];
  int64_t incl = run;
  for (int off = 1; off < kWave; off <<= 1) {
    const int64_t y = __shfl_up(incl, off, kWave);
    if (lane >= off) incl += y;
  }
  if (lane == kWave - 1) s_red[0][wave] = incl;
  __syncthreads();
  int64_t mu = incl - run;
  for (int q = 0; q < wave; q++) mu += s_red[0][q];
  // Eq. 2 per segment: M(U_{i-1}) + 2 M(V_i) + A(L_i)
  int64_t peak = 0;
  for (int c = c0; c < c1; c++) {
    const int64_t mem = mu + 2 * (int64_t)s_mv[c] + A[s_chain[c]];
    peak = mem > peak ? mem : peak;
    mu += s_gain[c];
  }
  peak = sched::wave_max(peak);
  tu = sched::wave_sum(tu);
  if (lane == 0) {
    s_red[1][wave] = peak;
    s_red[2][wave] = tu;
  }
  __syncthreads();
  if (tid == 0) {
    int64_t pk = 0, tsum = 0, mtot = 0;
    for (int q = 0; q < kWaves; q++) {
      pk = s_red[1][q] > pk ? s_red[1][q] : pk;
      tsum += s_red[2][q];
      mtot += s_red[0][q];
    }
    st->k = k;
    st->overhead = T_total - tsum;
    st->peak = pk;
    st->cache_mem = mtot;
  }
}

}  // namespace rcdp
