// Device helpers shared by the two wavefront DP fills (blocked.hip, ghost.hip).
//
// Both stream panel data global -> LDS with explicitly counted DMA loads,
// publish finished table cells with agent-coherent stores, and relax two
// 16-bit table cells per lane and instruction.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rc_internal.h"

namespace rcdp {
namespace wf {

constexpr int kWave = 64;
constexpr int kNB = 8;                   // panel records per pipeline stage

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Read-only inputs of a fill, read through the constant address space so
// that wave-uniform reads become scalar loads (they must not occupy the
// vector memory counter of the waves that count their DMA loads).
typedef const __attribute__((address_space(4))) int32_t cint32;
typedef const __attribute__((address_space(4))) int64_t cint64;
typedef const __attribute__((address_space(4))) uint64_t cu64;

// Global-memory pointers: the parameters of a batched launch come from
// memory, where the compiler no longer sees that they point to global
// memory; flat accesses would also count against the LDS counter that every
// barrier waits on.
typedef __attribute__((address_space(1))) int32_t gint32;
typedef __attribute__((address_space(1))) DevStatus gstatus;

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// 16 bytes per lane, global -> LDS at lds + 16 * lane, agent-coherent.  The
// load is invisible to the compiler's counter bookkeeping; every wait on it
// is explicit.  M0 (the LDS base of the copy) is saved and restored around it.
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
  uint32_t keep;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off sc1\n\ts_mov_b32 m0, %0"
      : "=&s"(keep)
      : "v"(g), "s"(lds)
      : "memory");
}

__device__ __forceinline__ void st_sc1(void* g, u32x2 v) {
  asm volatile("global_store_dwordx2 %0, %1, off sc1" : : "v"(g), "v"(v) : "memory");
}

__device__ __forceinline__ void st_sc1(void* g, u32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1" : : "v"(g), "v"(v) : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

__device__ __forceinline__ void wait_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

__device__ __forceinline__ int32_t ld_relaxed(const gint32* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ u16x2 as_u16x2(int32_t v) { return __builtin_bit_cast(u16x2, v); }

// The window DMA of one staged record for the column whose first computed
// cell lies at distance u0 from the row end and that computes cw cells: the
// window starts at table cell base + u0 and its 16-byte chunk kc is loaded
// when lo <= kc < hi (inside the source row's aligned slot, and the record
// reaches the column), else the infinity sentinel is.  The terms that do
// not depend on the column come precomputed with the record (words kRecDma
// ..), so a record costs a few scalar operations and two compares per lane.
struct WinDma {
  const uint16_t* base;
  int32_t lo, hi;
};

__device__ __forceinline__ WinDma win_dma(const int32_t* hd, bool valid, int32_t u0, int32_t cw,
                                          const uint16_t* m) {
  const int4 h = *reinterpret_cast<const int4*>(hd + kRecDma);
  const int2 g = *reinterpret_cast<const int2*>(hd + kRecDma + 4);
  const uint32_t blo = __builtin_amdgcn_readfirstlane(h.x);
  const int32_t bhi = __builtin_amdgcn_readfirstlane(h.y);
  const int32_t span = __builtin_amdgcn_readfirstlane(h.z);    // cells of the row's slot
  const int32_t er = __builtin_amdgcn_readfirstlane(h.w);      // emin - a
  const int32_t emin = __builtin_amdgcn_readfirstlane(g.x);
  const int32_t far = __builtin_amdgcn_readfirstlane(g.y);     // emax + P_i
  const bool live = valid && u0 + emin <= 0 && u0 + cw - 1 + far >= 0;
  const int32_t to_end = 1 - u0 - er;                          // cells from the window start to the row end
  WinDma w;
  w.base = m + ((((int64_t)bhi << 32) | blo) + u0);
  w.hi = live ? to_end >> 3 : 0;
  w.lo = (to_end - span) >> 3;
  return w;
}

// Two relaxations of Algorithm 1: m' = x + dm if x <= tau (tau = B - c, the
// budget test), else infinity, in packed unsigned 16-bit lanes with
// saturation.  y = x +sat dm; q = x -sat tau is nonzero exactly when the
// budget test fails, and q * 0xFFFF +sat y (one multiply-add with clamp) is
// then 0xFFFF, else y.  Every finite value stays below 0xFFFF, so the
// saturated value is the infinity code.
__device__ __forceinline__ u16x2 relax2(u16x2 acc, u16x2 x, u16x2 tau, u16x2 dm) {
  const u16x2 y = __builtin_elementwise_add_sat(x, dm);
  const u16x2 q = __builtin_elementwise_sub_sat(x, tau);
  u16x2 r;
  asm("v_pk_mad_u16 %0, %1, -1, %2 clamp" : "=v"(r) : "v"(q), "v"(y));
  return __builtin_elementwise_min(acc, r);
}

// The race test's delay (seed != 0): at one in four of the points a wave
// passes, it sleeps a pseudo-random 0..63 rounds, drawn from the seed, the
// column, the block and the point, so that the order in which columns and
// waves store, publish and poll changes from one seed to the next while the
// table must not.
__device__ __forceinline__ void jitter_delay(int32_t seed, int32_t c, int32_t b, int32_t point) {
  if (seed == 0) return;
  uint32_t h = (uint32_t)seed * 0x9E3779B1u ^ (uint32_t)c * 0x85EBCA77u ^
               (uint32_t)(b + 2) * 0xC2B2AE3Du ^ (uint32_t)point * 0x27D4EB2Fu;
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  h ^= h >> 12;
  h = __builtin_amdgcn_readfirstlane(h);
  if ((h & 3) != 0) return;
  for (uint32_t r = (h >> 2) & 63; r > 0; r--) __builtin_amdgcn_s_sleep(4);
}

// The parameters of table tk % nb of a batched launch, read through the
// constant address space so that they load into scalar registers like the
// kernel arguments of a single-table launch (nb == 1: p0 itself).
template <class P>
__device__ __forceinline__ P batch_params(const P& p0, const P* ps, int32_t nb, int32_t tk) {
  if (nb == 1) return p0;
  static_assert(sizeof(P) % 8 == 0, "parameter words");
  struct Words {
    uint64_t v[sizeof(P) / 8];
  } wd;
  cu64* const q = (cu64*)(ps + tk % nb);
#pragma unroll
  for (int i = 0; i < (int)(sizeof(P) / 8); i++) wd.v[i] = q[i];
  return __builtin_bit_cast(P, wd);
}

}  // namespace wf
}  // namespace rcdp
