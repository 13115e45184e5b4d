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

__device__ __forceinline__ int64_t wave_sum_i64(int64_t x) {
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, kWave);
  return x;
}

__device__ __forceinline__ int64_t word_cost(uint64_t bits, int word, const int32_t* c) {
  int64_t s = 0;
  while (bits) {
    s += c[word * 64 + __builtin_ctzll(bits)];
    bits &= bits - 1;
  }
  return s;
}

}  // namespace sched

// Every thread of the block calls it after the walk: chain[0 .. k) holds the
// chain from V back to its first set; it is written back in increasing order
// (L_1 .. L_k), seg[n] (segment index of each node), cached[n] (1 iff in U_k)
// and st->{k, overhead, peak, cache_mem} are filled.  s_chain[k] and s_M[n]
// are LDS scratch of the caller.
template <int kThreads>
__device__ __forceinline__ void finish_schedule(int32_t k, int n, int words, int64_t fstride,
                                const uint64_t* __restrict__ bits, const uint64_t* __restrict__ bd,
                                const int32_t* __restrict__ A, const int32_t* __restrict__ T,
                                const int32_t* __restrict__ M, int64_t T_total, DevStatus* st,
                                int32_t* chain, int32_t* seg, uint8_t* cached, int32_t* s_chain,
                                int32_t* s_M) {
  using sched::kWave;
  using sched::wave_sum_i64;
  using sched::word_cost;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  // chain in increasing order, kept in LDS as well; node memories in LDS
  for (int c = tid; c < k; c += kThreads) s_chain[c] = chain[k - 1 - c];
  for (int v = tid; v < n; v += kThreads) {
    seg[v] = -1;
    s_M[v] = M[v];
  }
  __syncthreads();
  for (int c = tid; c < k; c += kThreads) chain[c] = s_chain[c];
  if (tid >= kWave) return;
  // Eq. 2 per segment: M(U_{i-1}) + 2 M(V_i) + A(L_i), U grows by the
  // boundary of each L_i; the loads of kPre chain steps are issued together
  constexpr int kPre = 16;
  const bool active = lane < words;
  uint64_t U = 0, prev = 0;
  int64_t mu = 0, peak = 0;
  for (int c0 = 0; c0 < k; c0 += kPre) {
    uint64_t Ls[kPre], Bs[kPre];
    int32_t As[kPre];
#pragma unroll
    for (int x = 0; x < kPre; x++) {
      const int c = c0 + x < k ? c0 + x : k - 1;
      const int64_t sx = s_chain[c];
      Ls[x] = active ? bits[(int64_t)lane * fstride + sx] : 0ull;
      Bs[x] = active ? bd[(int64_t)lane * fstride + sx] : 0ull;
      As[x] = A[sx];
    }
#pragma unroll
    for (int x = 0; x < kPre; x++) {
      const int c = c0 + x;
      if (c >= k) break;
      const uint64_t Vi = Ls[x] & ~prev;
      const int64_t mv = wave_sum_i64(active ? word_cost(Vi, lane, s_M) : 0);
      const int64_t mem = mu + 2 * mv + As[x];
      peak = mem > peak ? mem : peak;
      for (uint64_t bb = Vi; bb; bb &= bb - 1) seg[lane * 64 + __builtin_ctzll(bb)] = c;
      const uint64_t add = Bs[x] & ~U;
      mu += wave_sum_i64(active ? word_cost(add, lane, s_M) : 0);
      U |= add;
      prev = Ls[x];
    }
  }
  for (int b = 0; b < 64 && active; b++) {
    const int v = lane * 64 + b;
    if (v < n) cached[v] = (uint8_t)((U >> b) & 1ull);
  }
  const int64_t tu = wave_sum_i64(active ? word_cost(U, lane, T) : 0);
  if (lane == 0) {
    st->k = k;
    st->overhead = T_total - tu;
    st->peak = peak;
    st->cache_mem = mu;
  }
}

}  // namespace rcdp
