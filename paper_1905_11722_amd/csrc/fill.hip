// The DP of Section 4.2 / Appendix A (Algorithm 1) on the device: table
// fill, selection of t*, traceback of optarg and re-evaluation of the
// resulting canonical strategy with Eq. 1 and Eq. 2.
//
// Table layout: one row per family member L, holding the cells
// t = 0 .. w_L - 1 (w_L = T(L \ boundary(L)) + 1; every cell beyond is
// provably infinite, since each recomputed node of a chain ending at L lies
// in L \ boundary(L)).  Rows are contiguous in t and end on 128-byte
// lines.  A cell stores m = opt[L, t] as uint16 (0xFFFF = infinity), or
// as uint32 (0xFFFFFFFF = infinity) for budgets beyond the 16-bit range
// (the level fill, selection, traceback and export take either width).
//
// Pull form of Algorithm 1: opt[L', t'] is the minimum over predecessors
// L (proper subsets of L' in the family) of opt[L, t' - dt] + dm, taken
// over the sources that pass the budget test opt[L, t] + c <= B.
//
// optarg is not stored by the fill.  Algorithm 1's strict update over
// ascending sources makes optarg[L', t'] the smallest family index L among
// the predecessors whose cell passes the budget test and reproduces
// opt[L', t'] (the first source to reach the minimum writes it, later ones
// only tie).  That rule is evaluated where optarg is needed: at every step
// of the traceback (k_trace) and, for a whole-table export, by k_arg_all.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>

#include "rc_internal.h"
#include "dominance.h"
#include "schedule.h"
#include "wavefront.h"

namespace rcdp {

namespace {

constexpr int kWave = 64;
constexpr int kFillThreads = 256;
constexpr int kCellsPerThread = 4;
constexpr int kTile = kFillThreads * kCellsPerThread;

// Infinity of a table of cells of type T.
template <class T>
__device__ __forceinline__ constexpr uint32_t cell_inf() {
  return sizeof(T) == 2 ? 0xFFFFu : 0xFFFFFFFFu;
}

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

// opt[empty, 0] = 0 (Algorithm 1's initial condition); selection state.
template <class T>
__global__ void k_solve_init(T* m, const int64_t* row_off, int objective, DevStatus* st) {
  if (threadIdx.x == 0) {
    m[row_off[0]] = 0;
    st->error = 0;
    st->t_sel = objective == RC_TIME_CENTRIC ? INT32_MAX : -1;
    st->m_sel = -1;
    st->k = 0;
  }
}

// One launch per size level (targets of equal size never contain each
// other).  Block (x, y): cells [x * kTile, (x + 1) * kTile) of target
// lb + y; each thread owns kCellsPerThread cells strided by the block size
// so that every source read and every store of a wave is contiguous.
// ws[i]: the source row's cells that may be read, t < ws[i] (its width w[i],
// or the end of its weak front under the dominance skip).
template <class T>
__global__ __launch_bounds__(kFillThreads) void k_fill_level(
    int64_t lb, const int32_t* __restrict__ w, const int64_t* __restrict__ row_off,
    const int64_t* __restrict__ pred_ptr, const int32_t* __restrict__ pidx,
    const int32_t* __restrict__ pdt, const int32_t* __restrict__ pdm,
    const int32_t* __restrict__ pc, int32_t Beff, const int32_t* __restrict__ ws,
    T* __restrict__ m) {
  const int64_t j = lb + blockIdx.y;
  const int32_t wj = w[j];
  const int32_t tile0 = blockIdx.x * kTile;
  if (tile0 >= wj) return;
  uint32_t acc[kCellsPerThread];
#pragma unroll
  for (int r = 0; r < kCellsPerThread; r++) acc[r] = cell_inf<T>();
  const int64_t p0 = pred_ptr[j], p1 = pred_ptr[j + 1];
  for (int64_t p = p0; p < p1; ++p) {
    // budget test of Algorithm 1: opt[L, t] + c <= B, i.e. opt[L, t] <= tau
    const int32_t tau = Beff - pc[p];
    if (tau < 0) continue;                    // no source cell can pass
    const int32_t dt = pdt[p];
    const int32_t i = pidx[p];
    const int32_t wi = ws[i];                 // cells of the source row that can be read
    if (dt >= tile0 + kTile || dt + wi <= tile0) continue;  // window misses the tile
    const T* src = m + row_off[i];
    const uint32_t dm = (uint32_t)pdm[p];
#pragma unroll
    for (int r = 0; r < kCellsPerThread; r++) {
      const int32_t t = tile0 + r * kFillThreads + (int32_t)threadIdx.x - dt;
      if ((uint32_t)t < (uint32_t)wi) {
        const uint32_t x = src[t];
        if (x <= (uint32_t)tau) acc[r] = min(acc[r], x + dm);
      }
    }
  }
  T* mo = m + row_off[j];
#pragma unroll
  for (int r = 0; r < kCellsPerThread; r++) {
    const int32_t tp = tile0 + r * kFillThreads + (int32_t)threadIdx.x;
    if (tp < wj) mo[tp] = (T)acc[r];
  }
}

// The level fill for 16-bit cells, eight cells per lane, two per packed
// instruction.  Cells are counted from the row's end, which lies on a
// kRowAlign boundary: lane group g of target j owns the cells at
// [E_j - 8 (g + 1), E_j - 8 g) (E_j = end of the row), one aligned 16-byte
// store, and the source cell of target cell x along a pair is x + D with
// D = row_off[i] - row_off[j] - dt, the same for every cell of the pair.
// So a pair's eight source cells start D mod 8 cells past an aligned
// 16-byte word: two aligned loads and a shift by that uniform amount.
// Source cells outside [0, ws[i]) and target cells before the row's first
// cell read as infinity.
//
// The NW waves of a workgroup own the same 512 cells and take every NW-th
// group of kLevelGroup pairs; their minima meet in LDS.  A group's
// records arrive in one vector load (word k on lane k) and are broadcast to
// scalar registers, then every source load of the group goes out before the
// first is used (a pair a lane skips loads the lane's own cells instead),
// so that a lane waits for memory twice per group, and the chain of groups
// a wave walks is 1/NW of the target's pairs.  With kFront the
// readable part of a source row is ws[i] (the dominance skip's front).
constexpr int kVecCells = 8;
constexpr int kVecTile = kWave * kVecCells;          // cells per workgroup
constexpr int kLevelGroup = 4;
static_assert(sizeof(LevelPair) == 32 && kLevelGroup * 8 <= 32, "a group's records on 32 lanes");

// words w[0..7] hold cells 0..15 of two aligned 16-byte loads; out[q] gets
// cells a + 2q and a + 2q + 1 (a uniform, 0..7)
template <int a>
__device__ __forceinline__ void take8(const uint32_t (&w)[8], uint32_t (&out)[4]) {
#pragma unroll
  for (int q = 0; q < 4; q++) {
    if (a % 2 == 0)
      out[q] = w[a / 2 + q];
    else
      out[q] = __builtin_amdgcn_alignbit(w[a / 2 + q + 1], w[a / 2 + q], 16);
  }
}

template <bool kFront, int NW>
__global__ __launch_bounds__(NW * kWave) void k_fill_level_vec(
    int64_t lb, const int32_t* __restrict__ w, const int64_t* __restrict__ row_off,
    const int64_t* __restrict__ pred_ptr, const LevelPair* __restrict__ lp, int32_t Beff,
    const int32_t* __restrict__ ws, uint16_t* __restrict__ m) {
  using wf::u16x2;
  constexpr int kLevelWaves = NW;
  __shared__ uint4 s_acc[kLevelWaves > 1 ? kLevelWaves - 1 : 1][kWave];
  const int64_t j = lb + blockIdx.y;
  const int32_t wj = w[j];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int64_t g = (int64_t)blockIdx.x * kWave + lane;
  // the group's first cell, as t of row j: wj - 8 (g + 1); nothing to store
  // when the whole group lies before t = 0.  Such a lane still runs the loop
  // (on the row's last group), since the records reach every lane of the wave
  // from lanes 0..31; a workgroup with no such lane leaves at once.
  const int64_t t_first = (int64_t)wj - kVecCells * (g + 1);
  const bool live = t_first + kVecCells > 0;
  if ((int64_t)wj - kVecCells * ((int64_t)blockIdx.x * kWave) <= 0) return;  // lane 0's group
  const int64_t rj = row_off[j];
  // the group's first cell (aligned: the row ends on a kRowAlign boundary)
  const int64_t dst = rj + wj - kVecCells * (live ? g + 1 : 1);
  uint32_t acc[4] = {0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};
  const int64_t p0 = pred_ptr[j], p1 = pred_ptr[j + 1];
  for (int64_t pg = p0 + (int64_t)wave * kLevelGroup; pg < p1;
       pg += (int64_t)kLevelWaves * kLevelGroup) {
    // the group's records (the array has kLevelGroup more at its end) in one
    // vector load, word k on lane k, then broadcast to scalar registers
    const int32_t word = reinterpret_cast<const int32_t*>(lp + pg)[lane & 31];
    LevelPair r[kLevelGroup];
#pragma unroll
    for (int q = 0; q < kLevelGroup; q++) {
      auto rd = [&](int k) { return __builtin_amdgcn_readlane(word, 8 * q + k); };
      r[q].lo = (int64_t)(((uint64_t)(uint32_t)rd(1) << 32) | (uint32_t)rd(0));
      r[q].base = (int64_t)(((uint64_t)(uint32_t)rd(3) << 32) | (uint32_t)rd(2));
      r[q].c = rd(4);
      r[q].dm = rd(5);
      r[q].w = rd(6);
      r[q].src = rd(7);
    }
    int64_t src[kLevelGroup], hi[kLevelGroup];
    bool use[kLevelGroup];
    uint4 v0[kLevelGroup], v1[kLevelGroup];
#pragma unroll
    for (int q = 0; q < kLevelGroup; q++) {
      // source cell of the group's first cell; readable cells [lo, hi)
      src[q] = dst - rj + r[q].base;
      hi[q] = r[q].lo + (kFront ? ws[r[q].src] : r[q].w);
      use[q] = pg + q < p1 && Beff - r[q].c >= 0 && src[q] + kVecCells > r[q].lo && src[q] < hi[q];
      const uint4* v = reinterpret_cast<const uint4*>(
          m + (use[q] ? src[q] - (src[q] & (kVecCells - 1)) : dst));
      v0[q] = v[0];
      v1[q] = v[1];
    }
#pragma unroll
    for (int q = 0; q < kLevelGroup; q++) {
      if (!use[q]) continue;
      const int32_t a = (int32_t)(src[q] & (kVecCells - 1));
      const uint32_t wd[8] = {v0[q].x, v0[q].y, v0[q].z, v0[q].w,
                              v1[q].x, v1[q].y, v1[q].z, v1[q].w};
      uint32_t x[4];
      switch (a) {
        case 0: take8<0>(wd, x); break;
        case 1: take8<1>(wd, x); break;
        case 2: take8<2>(wd, x); break;
        case 3: take8<3>(wd, x); break;
        case 4: take8<4>(wd, x); break;
        case 5: take8<5>(wd, x); break;
        case 6: take8<6>(wd, x); break;
        default: take8<7>(wd, x); break;
      }
      if (src[q] < r[q].lo || src[q] + kVecCells > hi[q]) {   // the row's edge: outside is infinite
#pragma unroll
        for (int c = 0; c < kVecCells; c++)
          if (src[q] + c < r[q].lo || src[q] + c >= hi[q]) x[c / 2] |= 0xFFFFu << (16 * (c % 2));
      }
      // budget test of Algorithm 1: opt[L, t] + c <= B, i.e. opt[L, t] <= tau
      const unsigned short tau = (unsigned short)(Beff - r[q].c);
      const unsigned short dm = (unsigned short)r[q].dm;
      const u16x2 tv = {tau, tau};
      const u16x2 dv = {dm, dm};
#pragma unroll
      for (int c = 0; c < 4; c++)
        acc[c] = __builtin_bit_cast(uint32_t, wf::relax2(__builtin_bit_cast(u16x2, acc[c]),
                                                         __builtin_bit_cast(u16x2, x[c]), tv, dv));
    }
  }
  // the waves' minima meet in LDS; wave 0 stores
  if (wave > 0) s_acc[wave - 1][lane] = make_uint4(acc[0], acc[1], acc[2], acc[3]);
  if (kLevelWaves > 1) __syncthreads();
  if (wave > 0 || !live) return;
#pragma unroll
  for (int q = 0; q < kLevelWaves - 1; q++) {
    const uint4 o = s_acc[q][lane];
    const uint32_t ov[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
    for (int c = 0; c < 4; c++)
      acc[c] = __builtin_bit_cast(uint32_t,
                                  __builtin_elementwise_min(__builtin_bit_cast(u16x2, acc[c]),
                                                            __builtin_bit_cast(u16x2, ov[c])));
  }
  if (t_first < 0) {                                 // cells before t = 0: padding, infinite
#pragma unroll
    for (int c = 0; c < kVecCells; c++)
      if (t_first + c < 0) acc[c / 2] |= 0xFFFFu << (16 * (c % 2));
  }
  *reinterpret_cast<uint4*>(m + dst) = make_uint4(acc[0], acc[1], acc[2], acc[3]);
}

// The level fill's record of each pair (built once per family).
__global__ void k_level_pairs(int64_t P, const int32_t* __restrict__ pidx,
                              const int32_t* __restrict__ pdt, const int32_t* __restrict__ pdm,
                              const int32_t* __restrict__ pc, const int32_t* __restrict__ w,
                              const int64_t* __restrict__ row_off, LevelPair* lp) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= P) return;
  const int32_t i = pidx[p];
  LevelPair r;
  r.lo = row_off[i];
  r.base = row_off[i] - pdt[p];
  r.c = pc[p];
  r.dm = pdm[p];
  r.w = w[i];
  r.src = i;
  lp[p] = r;
}

// The dominance skip of Section 4.2 (last paragraph) on finished rows
// lb + blockIdx.y: a cell t of row L is never propagated when an earlier
// cell of the same row holds strictly less memory.  Such a cell is stored as
// infinity, which leaves each row as its weak front (the cells with m no
// larger than every earlier m), the only cells that a later level, the
// selection of t* or the traceback reads.  we[L] = 1 + the last finite
// cell kept (0 when none): the level fill reads no source cell beyond it.
// Two passes over segments of kSeg cells, every (segment, row) a block:
// k_front_min stores each segment's least m, then k_front takes the least m
// of the segments before its own as the carry and scans its segment in
// chunks of kFillThreads cells, each cell read and rewritten by one thread.
constexpr int kSeg = 2048;

__global__ __launch_bounds__(kFillThreads) void k_front_min(
    int64_t lb, const int32_t* __restrict__ w, const int64_t* __restrict__ row_off,
    const uint16_t* __restrict__ m, int32_t nseg, uint32_t* __restrict__ segmin,
    int32_t* __restrict__ we) {
  __shared__ uint32_t s_wave[kFillThreads / kWave];
  const int64_t j = lb + blockIdx.y;
  const int32_t wj = w[j];
  const int32_t t0 = blockIdx.x * kSeg;
  const uint16_t* row = m + row_off[j];
  uint32_t x = kInfM;
  for (int32_t t = t0 + (int32_t)threadIdx.x; t < min(wj, t0 + kSeg); t += kFillThreads)
    x = min(x, (uint32_t)row[t]);
  for (int off = kWave / 2; off > 0; off >>= 1) x = min(x, (uint32_t)__shfl_xor(x, off, kWave));
  if (threadIdx.x % kWave == 0) s_wave[threadIdx.x / kWave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int q = 1; q < kFillThreads / kWave; q++) x = min(x, s_wave[q]);
    segmin[blockIdx.y * (int64_t)nseg + blockIdx.x] = x;
    if (blockIdx.x == 0) we[j] = 0;
  }
}

__global__ __launch_bounds__(kFillThreads) void k_front(
    int64_t lb, const int32_t* __restrict__ w, const int64_t* __restrict__ row_off,
    uint16_t* __restrict__ m, int32_t nseg, const uint32_t* __restrict__ segmin,
    int32_t* __restrict__ we) {
  __shared__ uint32_t s_wave[kFillThreads / kWave];
  __shared__ int32_t s_last;
  const int64_t j = lb + blockIdx.y;
  const int32_t wj = w[j];
  const int32_t s0 = blockIdx.x * kSeg;
  if (s0 >= wj) return;                     // the whole block leaves together
  const int32_t s1 = min(wj, s0 + kSeg);
  uint16_t* row = m + row_off[j];
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  if (threadIdx.x == 0) s_last = -1;
  uint32_t carry = kInfM;                   // least m of the earlier segments, then chunks
  for (int32_t q = 0; q < (int32_t)blockIdx.x; q++)
    carry = min(carry, segmin[blockIdx.y * (int64_t)nseg + q]);
  int32_t last = -1;
  for (int32_t c0 = s0; c0 < s1; c0 += kFillThreads) {
    const int32_t t = c0 + (int32_t)threadIdx.x;
    const uint32_t x = t < s1 ? row[t] : kInfM;
    uint32_t inc = x;                       // inclusive minimum along the wave
    for (int off = 1; off < kWave; off <<= 1) {
      const uint32_t y = __shfl_up(inc, off, kWave);
      if (lane >= off) inc = min(inc, y);
    }
    uint32_t exc = __shfl_up(inc, 1, kWave);
    if (lane == 0) exc = kInfM;
    if (lane == kWave - 1) s_wave[wave] = inc;
    __syncthreads();
    uint32_t before = carry;                // earlier chunks and earlier waves
    for (int q = 0; q < wave; q++) before = min(before, s_wave[q]);
    uint32_t chunk = carry;
    for (int q = 0; q < kFillThreads / kWave; q++) chunk = min(chunk, s_wave[q]);
    __syncthreads();                        // s_wave is rewritten by the next chunk
    const uint32_t least = min(before, exc);
    if (t < s1) {
      const bool keep = x != kInfM && x <= least;
      if (!keep && x != kInfM) row[t] = (uint16_t)kInfM;
      if (keep) last = t;
    }
    carry = chunk;
  }
  if (last >= 0) atomicMax(&s_last, last);
  __syncthreads();
  if (threadIdx.x == 0 && s_last >= 0) atomicMax(&we[j], s_last + 1);
}

// optarg of every cell of targets [lb, lb + gridDim.y) from the final
// table: the smallest predecessor index whose cell passes the budget test
// and reproduces the target value (Algorithm 1's first writer).
template <class T>
__global__ __launch_bounds__(kFillThreads) void k_arg_all(
    int64_t lb, const int32_t* __restrict__ w, const int64_t* __restrict__ row_off,
    const int64_t* __restrict__ pred_ptr, const int32_t* __restrict__ pidx,
    const int32_t* __restrict__ pdt, const int32_t* __restrict__ pdm,
    const int32_t* __restrict__ pc, int32_t Beff, const T* __restrict__ m,
    uint16_t* __restrict__ arg) {
  const int64_t j = lb + blockIdx.y;
  const int32_t wj = w[j];
  const int32_t tp = blockIdx.x * kFillThreads + threadIdx.x;
  if (tp >= wj) return;
  const uint32_t mj = m[row_off[j] + tp];
  uint32_t a = kNoArg;
  if (mj != cell_inf<T>() && j > 0) {
    for (int64_t p = pred_ptr[j]; p < pred_ptr[j + 1]; ++p) {
      const int32_t t = tp - pdt[p];
      const int32_t i = pidx[p];
      if ((uint32_t)t >= (uint32_t)w[i]) continue;
      const uint32_t x = m[row_off[i] + t];
      if (x != cell_inf<T>() && (int64_t)x <= (int64_t)Beff - pc[p] &&
          (uint32_t)(x + pdm[p]) == mj) {
        a = (uint32_t)i;
        break;
      }
    }
  }
  arg[row_off[j] + tp] = (uint16_t)a;
}

// t* = min (time-centric) or max (memory-centric) finite t of row V.
// A few workgroups stride over the row, reduce within the wave and then the
// workgroup, and issue one atomic each (one atomic per wave serialised on
// the one address).
constexpr int kSelectThreads = 256;
constexpr int kSelectBlocks = 64;

template <class T>
__global__ __launch_bounds__(kSelectThreads) void k_select(const T* m, const int64_t* row_off,
                                                          int64_t v, const int32_t* w,
                                                          int objective, DevStatus* st) {
  __shared__ int32_t s_best[kSelectThreads / kWave];
  const int64_t off = row_off[v];
  const int32_t wv = w[v];
  const bool tc = objective == RC_TIME_CENTRIC;
  int32_t best = tc ? INT32_MAX : -1;
  for (int32_t t = blockIdx.x * blockDim.x + threadIdx.x; t < wv; t += gridDim.x * blockDim.x)
    if (m[off + t] != cell_inf<T>()) best = tc ? min(best, t) : max(best, t);
  for (int o = kWave / 2; o > 0; o >>= 1) {
    const int32_t y = __shfl_xor(best, o, kWave);
    best = tc ? min(best, y) : max(best, y);
  }
  if ((threadIdx.x & (kWave - 1)) == 0) s_best[threadIdx.x / kWave] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int q = 1; q < kSelectThreads / kWave; q++)
      best = tc ? min(best, s_best[q]) : max(best, s_best[q]);
    if (tc ? best != INT32_MAX : best >= 0) {
      if (tc)
        atomicMin(&st->t_sel, best);
      else
        atomicMax(&st->t_sel, best);
    }
  }
}

template <class T>
__global__ void k_select_finish(const T* m, const int64_t* row_off, int64_t v, DevStatus* st) {
  if (threadIdx.x != 0) return;
  if (st->t_sel == INT32_MAX) st->t_sel = -1;
  st->m_sel = st->t_sel >= 0 ? (int32_t)m[row_off[v] + st->t_sel] : -1;
}

// Traceback from (V, t*) (Section 4.2), then Eq. 1 and Eq. 2 of the chain
// from their definitions: U_i is the union of boundaries of L_1..L_i,
// segment i needs M(U_{i-1}) + 2 M(V_i) + A(L_i), the overhead is
// T(V \ U_k).  At each step the workgroup scans the predecessors of L'
// (ascending family index, kTraceThreads at a time) for optarg[L', t']:
// the smallest index whose cell passes the budget test and reproduces the
// target value.  The re-evaluation runs on wave 0, lane w holding word w.
constexpr int kTraceThreads = 512;
constexpr int kTraceLds = 2048;       // families up to this size keep their per-set arrays in LDS

template <bool kLds, class Cell>
__global__ __launch_bounds__(kTraceThreads) void k_trace(
    int64_t F, int n, int words, int64_t fstride, const uint64_t* __restrict__ bits,
    const uint64_t* __restrict__ bd, const int32_t* __restrict__ A, const int32_t* __restrict__ T,
    const int32_t* __restrict__ M, const int32_t* __restrict__ w,
    const int64_t* __restrict__ row_off, const int64_t* __restrict__ pred_ptr,
    const int32_t* __restrict__ pidx, const int32_t* __restrict__ pdt,
    const int32_t* __restrict__ pdm, const int32_t* __restrict__ pc, int32_t Beff,
    const Cell* __restrict__ m, int64_t T_total, DevStatus* st, int32_t* chain, int32_t* seg,
    uint8_t* cached) {
  // per-set arrays of small families live in LDS for the whole walk
  __shared__ int32_t s_w[kTraceLds];
  __shared__ int64_t s_off[kTraceLds];
  __shared__ int64_t s_pp[kTraceLds + 1];
  // per chunk of predecessors, alternating by parity: the first hit of each
  // wave and every thread's (source, dt)
  __shared__ int32_t s_first[2][kTraceThreads / kWave];
  __shared__ int32_t s_src[2][kTraceThreads];
  __shared__ int32_t s_dt[2][kTraceThreads];
  __shared__ int32_t s_chain[kMaxNodes + 1];        // a chain adds a node per step
  __shared__ int32_t s_M[kMaxNodes];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  if (kLds) {
    for (int64_t x = tid; x < F; x += kTraceThreads) {
      s_w[x] = w[x];
      s_off[x] = row_off[x];
      s_pp[x] = pred_ptr[x];
    }
    if (tid == 0) s_pp[F] = pred_ptr[F];
  }
  // Every step of the walk reads the predecessor lists of one set: bring
  // them all into this CU's L2 first when they are small (a few MB), so that
  // those reads cost an L2 hit instead of a trip to memory.
  const int64_t P = pred_ptr[F];
  if (P <= ((int64_t)1 << 17)) {
    int32_t acc = 0;
    for (int64_t x = tid * 16; x < P; x += kTraceThreads * 16)
      acc ^= pidx[x] ^ pdt[x] ^ pc[x] ^ pdm[x];
    if (acc == 0x7fffffff) st->pad0 = acc;          // keeps the loads
  }
  __syncthreads();
  auto Wd = [&](int64_t i) { return kLds ? s_w[i] : w[i]; };
  auto Off = [&](int64_t i) { return kLds ? s_off[i] : row_off[i]; };
  auto PP = [&](int64_t i) { return kLds ? s_pp[i] : pred_ptr[i]; };

  // The walk is identical in every thread; only the predecessor scan is split.
  int64_t j = F - 1;
  int64_t t = st->t_sel;
  int32_t k = 0;
  bool bad = t < 0;
  int par = 0;
  while (j != 0 && !bad) {
    if (t < 0 || t >= Wd(j) || k >= F || k > n) {     // each step removes a node
      bad = true;
      break;
    }
    const int64_t p0 = PP(j), p1 = PP(j + 1);
    const uint32_t mj = m[Off(j) + t];
    int32_t next_i = -1, next_dt = 0;
    for (int64_t base = p0; base < p1 && next_i < 0; base += kTraceThreads) {
      // every load of a chunk is issued unconditionally (a thread past the
      // list reads the list's first pair, a source cell out of its row reads
      // the row's first cell) and the tests come last, so a step waits for
      // the pair data, the source rows' extents and the source cells only
      const int64_t p = base + tid;
      const bool valid = p < p1;
      const int64_t pq = valid ? p : p0;
      const int32_t i = pidx[pq], dt = pdt[pq], c = pc[pq], dm = pdm[pq];
      const int64_t ts = t - dt;
      const bool inrow = valid && ts >= 0 && ts < Wd(i);
      const uint32_t x = m[Off(i) + (inrow ? ts : 0)];
      const bool hit = inrow && x != cell_inf<Cell>() && (int64_t)x <= (int64_t)Beff - c &&
                       (uint32_t)(x + dm) == mj;
      const unsigned long long bal = __ballot(hit);
      if (lane == 0) s_first[par][wave] = bal ? wave * kWave + __ffsll((long long)bal) - 1 : INT32_MAX;
      s_src[par][tid] = i;
      s_dt[par][tid] = dt;
      __syncthreads();
      int32_t f = INT32_MAX;
#pragma unroll
      for (int q = 0; q < kTraceThreads / kWave; q++) f = min(f, s_first[par][q]);
      if (f != INT32_MAX) {                    // the smallest predecessor index that hits
        next_i = s_src[par][f];
        next_dt = s_dt[par][f];
      }
      par ^= 1;
    }
    if (next_i < 0 || mj == cell_inf<Cell>()) {
      bad = true;
      break;
    }
    if (tid == 0) chain[k] = (int32_t)j;
    k++;
    t -= next_dt;
    j = next_i;
  }
  if (t != 0) bad = true;                            // the walk must end at (empty, 0)
  __syncthreads();
  if (bad) {
    if (tid == 0) {
      st->error = 2;
      st->k = -1;
    }
    return;
  }
  finish_schedule<kTraceThreads>(k, n, words, fstride, bits, bd, A, T, M, T_total, st, chain, seg,
                                  cached, s_chain, s_M);
}

// The traceback through an optarg slice.  When t* is small, every step of
// the walk stays among the cells (L', t') with t' <= t*: optarg of all of
// them (by the rule of k_trace) is evaluated at once, over the whole chip,
// and the walk then follows it, one load per step instead of a scan of the
// predecessor list.  k_trace_args: workgroup (x, L') takes the 64 cells
// t' = 64 x + lane of row L', its waves the predecessor list in interleaved
// groups of 64 pairs (group g to wave g mod kArgWaves).  Each lane keeps the
// first hit of its wave, and the least over the waves is the first hit of
// the list.  A wave stops when every lane has a hit: its later groups hold
// only larger indices.  The result of cell (L', t') is nxt[L' S + t'] =
// L | (t' - dt) << 16 (S = t* + 1 <= 65536, family indices below 65535), or
// kNoNext: no hit, infinite, L' empty or t' beyond the row.
constexpr int kArgWaves = 4;
constexpr uint32_t kNoNext = 0xFFFFFFFFu;

template <class Cell>
__global__ __launch_bounds__(kArgWaves* kWave) void k_trace_args(
    int32_t S, const int32_t* __restrict__ w, const int64_t* __restrict__ row_off,
    const int64_t* __restrict__ pred_ptr, const int32_t* __restrict__ pidx,
    const int32_t* __restrict__ pdt, const int32_t* __restrict__ pdm,
    const int32_t* __restrict__ pc, int32_t Beff, const Cell* __restrict__ m,
    uint32_t* __restrict__ nxt) {
  __shared__ int32_t s_hit[kArgWaves][kWave];
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int64_t j = blockIdx.y;
  const int32_t t = blockIdx.x * kWave + lane;
  const int32_t wj = w[j];
  const uint32_t mj = m[row_off[j] + (t < wj ? t : 0)];
  const bool need = j > 0 && t < S && t < wj && mj != cell_inf<Cell>();
  const int64_t p0 = pred_ptr[j], p1 = pred_ptr[j + 1];
  int32_t hit = INT32_MAX;
  if (__any(need)) {
    for (int64_t g = p0 + (int64_t)wave * kWave; g < p1; g += kArgWaves * kWave) {
      // lane l holds pair g + l: the source row's cell of target t at
      // base + t, in the row when t - dt lies in [0, w_L); past the list w = 0
      const int64_t p = g + lane;
      const int64_t pq = p < p1 ? p : p0;
      const int32_t i = pidx[pq], dt = pdt[pq], c = pc[pq], dm = pdm[pq];
      const int64_t base = row_off[i] - dt;
      const int32_t wi = p < p1 ? w[i] : 0;
      const uint32_t blo = (uint32_t)base, bhi = (uint32_t)((uint64_t)base >> 32);
      const int32_t cnt = (int32_t)std::min<int64_t>(kWave, p1 - g);
      for (int32_t k0 = 0; k0 < cnt; k0 += 8) {
        // eight source cells loaded before any test (a cell outside its row
        // is read at the row's first cell and not used)
        uint32_t x[8];
        bool in[8];
#pragma unroll
        for (int u = 0; u < 8; u++) {
          const int k = k0 + u;
          const int32_t dtk = __builtin_amdgcn_readlane(dt, k);
          const int32_t wk = __builtin_amdgcn_readlane(wi, k);
          const int64_t bk = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane(bhi, k) << 32) |
                                       (uint32_t)__builtin_amdgcn_readlane(blo, k));
          in[u] = (uint32_t)(t - dtk) < (uint32_t)wk;
          x[u] = m[bk + (in[u] ? t : dtk)];
        }
#pragma unroll
        for (int u = 0; u < 8; u++) {
          const int k = k0 + u;
          const int32_t ck = __builtin_amdgcn_readlane(c, k);
          const int32_t dmk = __builtin_amdgcn_readlane(dm, k);
          if (hit == INT32_MAX && in[u] && x[u] != cell_inf<Cell>() &&
              (int64_t)x[u] <= (int64_t)Beff - ck && (uint32_t)(x[u] + dmk) == mj)
            hit = (int32_t)(g - p0) + k;
        }
      }
      if (!__any(need && hit == INT32_MAX)) break;
    }
  }
  s_hit[wave][lane] = need ? hit : INT32_MAX;
  __syncthreads();
  if (wave != 0 || t >= S) return;
  int32_t h = INT32_MAX;
#pragma unroll
  for (int q = 0; q < kArgWaves; q++) h = min(h, s_hit[q][lane]);
  uint32_t e = kNoNext;
  if (h != INT32_MAX) {
    const int64_t p = p0 + h;
    e = (uint32_t)pidx[p] | ((uint32_t)(t - pdt[p]) << 16);
  }
  nxt[j * S + t] = e;
}

// The walk over the slice of k_trace_args from (V, t*), then Eq. 1 and
// Eq. 2 of the chain as in k_trace.  Thread 0 walks; meanwhile the other
// waves read the slice from its last row down (the order of the walk), so
// that most of the walk's loads hit the L2 of the XCD it runs on.
__global__ __launch_bounds__(kTraceThreads) void k_trace_follow(
    int64_t F, int n, int words, int64_t fstride, const uint64_t* __restrict__ bits,
    const uint64_t* __restrict__ bd, const int32_t* __restrict__ A, const int32_t* __restrict__ T,
    const int32_t* __restrict__ M, int32_t S, const uint32_t* __restrict__ nxt, int64_t T_total,
    DevStatus* st, int32_t* chain, int32_t* seg, uint8_t* cached) {
  __shared__ int32_t s_chain[kMaxNodes + 1];
  __shared__ int32_t s_M[kMaxNodes];
  __shared__ int32_t s_k;
  const int tid = threadIdx.x;
  if (tid >= kWave) {
    // eight loads in flight per lane
    constexpr int64_t kStride = kTraceThreads - kWave;
    const uint4* q = reinterpret_cast<const uint4*>(nxt);
    uint32_t acc = 0;
    int64_t x = F * S / 4 - 1 - (tid - kWave);
    for (; x >= 7 * kStride; x -= 8 * kStride) {
      uint4 v[8];
#pragma unroll
      for (int u = 0; u < 8; u++) v[u] = q[x - u * kStride];
#pragma unroll
      for (int u = 0; u < 8; u++) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; x >= 0; x -= kStride) {
      const uint4 v = q[x];
      acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x7fffffffu) st->pad0 = (int32_t)acc;   // keeps the loads
  } else if (tid == 0) {
    int64_t j = F - 1;
    int32_t t = st->t_sel;
    int32_t k = 0;
    bool bad = t < 0 || t >= S;
    while (!bad && j != 0) {
      if (k >= F || k > n) {                      // each step removes a node
        bad = true;
        break;
      }
      const uint32_t e = nxt[j * S + t];
      if (e == kNoNext) {
        bad = true;
        break;
      }
      chain[k++] = (int32_t)j;
      j = e & 0xFFFFu;
      t = (int32_t)(e >> 16);
    }
    if (t != 0) bad = true;                        // the walk must end at (empty, 0)
    s_k = bad ? -1 : k;
  }
  __syncthreads();
  const int32_t k = s_k;
  if (k < 0) {
    if (tid == 0) {
      st->error = 2;
      st->k = -1;
    }
    return;
  }
  finish_schedule<kTraceThreads>(k, n, words, fstride, bits, bd, A, T, M, T_total, st, chain, seg,
                                  cached, s_chain, s_M);
}

}  // namespace

hipError_t launch_solve_init(rc_solution sol, hipStream_t s) {
  rc_family f = sol->f;
  if (sol->cell32)
    hipLaunchKernelGGL(k_solve_init<uint32_t>, dim3(1), dim3(64), 0, s, sol->m32, f->row_off,
                       sol->objective, sol->status);
  else
    hipLaunchKernelGGL(k_solve_init<uint16_t>, dim3(1), dim3(64), 0, s, sol->m, f->row_off,
                       sol->objective, sol->status);
  return hipGetLastError();
}

// Waves per workgroup of a level of the 16-bit level fill: enough that each
// walks at most two groups of the level's longest pair list (1 to 16), but
// no more than keep eight waves per SIMD busy: wide rows already fill the
// chip with workgroups, and their levels are bound by the source reads.
template <bool kFront>
static void launch_level_vec(rc_family f, int64_t l, dim3 grid, int64_t lb, int32_t Beff,
                             const int32_t* ws, uint16_t* m, hipStream_t s) {
  const int64_t most = f->level_pairs[l];
  const int64_t blocks = (int64_t)grid.x * grid.y;
  const int64_t cap = 8 * 4 * (int64_t)num_cus();        // eight waves per SIMD
  int nw = 1;
  while (nw < 16 && (int64_t)nw * 2 * kLevelGroup < most) nw *= 2;
  while (nw > 1 && blocks * nw > cap) nw /= 2;
#define RCDP_LEVEL_VEC(NW)                                                                  \
  hipLaunchKernelGGL((k_fill_level_vec<kFront, NW>), grid, dim3(NW * kWave), 0, s, lb, f->w, \
                     f->row_off, f->pred_ptr, f->lpair, Beff, ws, m)
  switch (nw) {
    case 1: RCDP_LEVEL_VEC(1); break;
    case 2: RCDP_LEVEL_VEC(2); break;
    case 4: RCDP_LEVEL_VEC(4); break;
    case 8: RCDP_LEVEL_VEC(8); break;
    default: RCDP_LEVEL_VEC(16); break;
  }
#undef RCDP_LEVEL_VEC
}

template <class T>
static void fill_levels(rc_solution sol, T* m, hipStream_t s) {
  rc_family f = sol->f;
  const int64_t L = (int64_t)f->level_ptr.size() - 1;
  for (int64_t l = 1; l < L; l++) {            // level 0 is the empty set
    const int64_t lb = f->level_ptr[l], le = f->level_ptr[l + 1];
    if (le <= lb) continue;
    if (sizeof(T) == 2) {
      const int64_t tiles = (f->level_maxw[l] + kVecTile - 1) / kVecTile;
      if (tiles <= 0) continue;
      launch_level_vec<false>(f, l, dim3((unsigned)tiles, (unsigned)(le - lb)), lb,
                              (int32_t)sol->Beff, f->w, reinterpret_cast<uint16_t*>(m), s);
    } else {
      const int64_t tiles = (f->level_maxw[l] + kTile - 1) / kTile;
      if (tiles <= 0) continue;
      hipLaunchKernelGGL(k_fill_level<T>, dim3((unsigned)tiles, (unsigned)(le - lb)),
                         dim3(kFillThreads), 0, s, lb, f->w, f->row_off, f->pred_ptr, f->pidx,
                         f->pdt, f->pdm, f->pc, (int32_t)sol->Beff, f->w, m);
    }
  }
}

// The family's level-fill pair records, built by its first level fill.
static hipError_t ensure_level_pairs(rc_family f, hipStream_t s) {
  if (f->lpair || f->P == 0) return hipSuccess;
  f->lpair = f->arena.get_n<LevelPair>(f->P + kLevelGroup);   // a group may read past the end
  if (!f->lpair) return hipErrorOutOfMemory;
  hipError_t e = hipMemsetAsync(f->lpair + f->P, 0, sizeof(LevelPair) * kLevelGroup, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_level_pairs, dim3((unsigned)((f->P + 255) / 256)), dim3(256), 0, s, f->P,
                     f->pidx, f->pdt, f->pdm, f->pc, f->w, f->row_off, f->lpair);
  return hipGetLastError();
}

hipError_t launch_fill(rc_solution sol, hipStream_t s) {
  if (sol->cell32) {
    fill_levels(sol, sol->m32, s);
  } else {
    const hipError_t e = ensure_level_pairs(sol->f, s);
    if (e != hipSuccess) return e;
    fill_levels(sol, sol->m, s);
  }
  return hipGetLastError();
}

hipError_t launch_fill_dominance(rc_solution sol, int32_t* we, hipStream_t s) {
  rc_family f = sol->f;
  const hipError_t le = ensure_level_pairs(f, s);
  if (le != hipSuccess) return le;
  const int64_t L = (int64_t)f->level_ptr.size() - 1;
  int64_t most = 1;                         // segment minima of the largest level
  for (int64_t l = 0; l < L; l++)
    most = std::max<int64_t>(most, (f->level_ptr[l + 1] - f->level_ptr[l]) *
                                       ((f->level_maxw[l] + kSeg - 1) / kSeg));
  uint32_t* segmin = sol->arena.get_n<uint32_t>(most);
  if (!segmin) return hipErrorOutOfMemory;
  auto front = [&](int64_t lb, int64_t rows, int32_t maxw) {
    const int32_t nseg = std::max<int32_t>(1, (maxw + kSeg - 1) / kSeg);
    const dim3 grid((unsigned)nseg, (unsigned)rows);
    hipLaunchKernelGGL(k_front_min, grid, dim3(kFillThreads), 0, s, lb, f->w, f->row_off,
                       (const uint16_t*)sol->m, nseg, segmin, we);
    hipLaunchKernelGGL(k_front, grid, dim3(kFillThreads), 0, s, lb, f->w, f->row_off, sol->m,
                       nseg, (const uint32_t*)segmin, we);
  };
  front(0, 1, f->level_maxw[0]);            // the empty set
  for (int64_t l = 1; l < L; l++) {
    const int64_t lb = f->level_ptr[l], le = f->level_ptr[l + 1];
    const int64_t tiles = (f->level_maxw[l] + kVecTile - 1) / kVecTile;
    if (tiles <= 0 || le <= lb) continue;
    launch_level_vec<true>(f, l, dim3((unsigned)tiles, (unsigned)(le - lb)), lb,
                           (int32_t)sol->Beff, (const int32_t*)we, sol->m, s);
    front(lb, le - lb, f->level_maxw[l]);
  }
  return hipGetLastError();
}

template <class T>
static void select_t(rc_solution sol, const T* m, hipStream_t s) {
  rc_family f = sol->f;
  const int64_t v = f->F - 1;
  const int64_t wv = f->w_host[v];
  const unsigned blocks =
      (unsigned)std::min<int64_t>((wv + kSelectThreads - 1) / kSelectThreads, kSelectBlocks);
  hipLaunchKernelGGL(k_select<T>, dim3(blocks > 0 ? blocks : 1), dim3(kSelectThreads), 0, s, m,
                     f->row_off, v, f->w, sol->objective, sol->status);
  hipLaunchKernelGGL(k_select_finish<T>, dim3(1), dim3(64), 0, s, m, f->row_off, v, sol->status);
}

hipError_t launch_select(rc_solution sol, hipStream_t s) {
  if (sol->cell32)
    select_t<uint32_t>(sol, sol->m32, s);
  else
    select_t<uint16_t>(sol, sol->m, s);
  return hipGetLastError();
}

// The slice traceback is taken when its evaluation, about (t* + 1) P pair
// tests spread over the chip, costs less than the longest walk the scan
// could take, and its slice of 4 (t* + 1) F bytes is small; otherwise the
// scan of k_trace.  Measured here: a scan step costs about 0.8 us, the
// slice's tests run at about 5e11 per second (so 4e5 tests per step of the
// longest chain, min(F - 1, n) steps), and its walk costs about 0.2 us a
// step.  RCDP_TRACE = scan | slice forces one (slice within its size limits).
constexpr int64_t kSliceTests = (int64_t)1 << 26;
constexpr int64_t kSliceTestsPerStep = 400000;
constexpr int64_t kSliceCells = (int64_t)1 << 24;

static bool use_slice(rc_solution sol) {
  rc_family f = sol->f;
  const int64_t S = sol->t_star + 1;
  if (sol->t_star < 0 || S > 65536 || f->F >= 65535 || f->F * S > kSliceCells) return false;
  const char* env = std::getenv("RCDP_TRACE");
  if (env && std::strcmp(env, "scan") == 0) return false;
  if (env && std::strcmp(env, "slice") == 0) return true;
  const int64_t steps = std::min<int64_t>(f->F - 1, f->g->n);
  return S * f->P <= std::min<int64_t>(kSliceTests, kSliceTestsPerStep * steps);
}

template <class T>
static hipError_t trace_t(rc_solution sol, const T* m, hipStream_t s) {
  rc_family f = sol->f;
  rc_graph g = f->g;
  sol->trace_path = use_slice(sol) ? 1 : 0;
  if (sol->trace_path == 1) {
    const int32_t S = (int32_t)(sol->t_star + 1);
    const int64_t cells = f->F * (int64_t)S;
    if (sol->nxt_cells < cells) {
      sol->nxt = sol->arena.get_n<uint32_t>(cells);
      if (!sol->nxt) return hipErrorOutOfMemory;
      sol->nxt_cells = cells;
    }
    hipLaunchKernelGGL(k_trace_args<T>, dim3((unsigned)((S + kWave - 1) / kWave), (unsigned)f->F),
                       dim3(kArgWaves * kWave), 0, s, S, f->w, f->row_off, f->pred_ptr, f->pidx,
                       f->pdt, f->pdm, f->pc, (int32_t)sol->Beff, m, sol->nxt);
    hipLaunchKernelGGL(k_trace_follow, dim3(1), dim3(kTraceThreads), 0, s, f->F, g->n, g->words,
                       f->fstride, f->bits, f->bd, f->A, g->dT, g->dM, S, sol->nxt, g->T_total,
                       sol->status, sol->chain, sol->seg, sol->cached);
  } else if (f->F <= kTraceLds) {
    hipLaunchKernelGGL((k_trace<true, T>), dim3(1), dim3(kTraceThreads), 0, s, f->F, g->n, g->words,
                       f->fstride, f->bits, f->bd, f->A, g->dT, g->dM, f->w, f->row_off,
                       f->pred_ptr, f->pidx, f->pdt, f->pdm, f->pc, (int32_t)sol->Beff, m,
                       g->T_total, sol->status, sol->chain, sol->seg, sol->cached);
  } else {
    hipLaunchKernelGGL((k_trace<false, T>), dim3(1), dim3(kTraceThreads), 0, s, f->F, g->n,
                       g->words, f->fstride, f->bits, f->bd, f->A, g->dT, g->dM, f->w,
                       f->row_off, f->pred_ptr, f->pidx, f->pdt, f->pdm, f->pc,
                       (int32_t)sol->Beff, m, g->T_total, sol->status, sol->chain, sol->seg,
                       sol->cached);
  }
  return hipGetLastError();
}

hipError_t launch_trace(rc_solution sol, hipStream_t s) {
  return sol->cell32 ? trace_t<uint32_t>(sol, sol->m32, s) : trace_t<uint16_t>(sol, sol->m, s);
}

template <class T>
static void arg_all_t(rc_solution sol, const T* m, hipStream_t s) {
  rc_family f = sol->f;
  const int64_t L = (int64_t)f->level_ptr.size() - 1;
  for (int64_t l = 0; l < L; l++) {
    const int64_t lb = f->level_ptr[l], le = f->level_ptr[l + 1];
    const int64_t tiles = (f->level_maxw[l] + kFillThreads - 1) / kFillThreads;
    if (tiles <= 0 || le <= lb) continue;
    hipLaunchKernelGGL(k_arg_all<T>, dim3((unsigned)tiles, (unsigned)(le - lb)),
                       dim3(kFillThreads), 0, s, lb, f->w, f->row_off, f->pred_ptr, f->pidx,
                       f->pdt, f->pdm, f->pc, (int32_t)sol->Beff, m, sol->arg);
  }
}

hipError_t launch_arg_all(rc_solution sol, hipStream_t s) {
  if (sol->cell32)
    arg_all_t<uint32_t>(sol, sol->m32, s);
  else
    arg_all_t<uint16_t>(sol, sol->m, s);
  return hipGetLastError();
}

}  // namespace rcdp
