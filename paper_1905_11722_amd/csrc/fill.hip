// The DP of Section 4.2 / Appendix A (Algorithm 1) on the device: table
// fill, selection of t*, traceback of optarg and re-evaluation of the
// resulting canonical strategy with Eq. 1 and Eq. 2.
//
// Table layout: one row per family member L, holding the cells
// t = 0 .. w_L - 1 (w_L = T(L \ boundary(L)) + 1; every cell beyond is
// provably infinite, since each recomputed node of a chain ending at L lies
// in L \ boundary(L)).  Rows are contiguous in t and start on 128-byte lines.
// A cell stores m = opt[L, t] as uint16 (0xFFFF = infinity) and optarg as the
// uint16 family index of the predecessor.
//
// Pull form of Algorithm 1: opt[L', t'] is the minimum over predecessors
// L (proper subsets of L' in the family) of opt[L, t' - dt] + dm, taken
// over the sources that pass the budget test opt[L, t] + c <= B.  The
// strict update of Algorithm 1, which visits sources in ascending family
// index, keeps the first (smallest-index) source among equal minima; the
// kernel reproduces that with one unsigned minimum over the packed key
// (m' << 16) | index(L).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "rc_internal.h"

namespace rcdp {

namespace {

constexpr int kWave = 64;
constexpr int kFillThreads = 256;
constexpr int kCellsPerThread = 4;
constexpr int kTile = kFillThreads * kCellsPerThread;

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
__global__ void k_solve_init(uint16_t* m, uint16_t* arg, const int64_t* row_off, int objective,
                             DevStatus* st) {
  if (threadIdx.x == 0) {
    m[row_off[0]] = 0;
    arg[row_off[0]] = (uint16_t)kNoArg;
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
__global__ __launch_bounds__(kFillThreads) void k_fill_level(
    int64_t lb, const int32_t* __restrict__ w, const int64_t* __restrict__ row_off,
    const int64_t* __restrict__ pred_ptr, const int32_t* __restrict__ pidx,
    const int32_t* __restrict__ pdt, const int32_t* __restrict__ pdm,
    const int32_t* __restrict__ pc, int32_t Beff, uint16_t* __restrict__ m,
    uint16_t* __restrict__ arg) {
  const int64_t j = lb + blockIdx.y;
  const int32_t wj = w[j];
  const int32_t tile0 = blockIdx.x * kTile;
  if (tile0 >= wj) return;
  uint32_t acc[kCellsPerThread];
#pragma unroll
  for (int r = 0; r < kCellsPerThread; r++) acc[r] = 0xFFFFFFFFu;
  const int64_t p0 = pred_ptr[j], p1 = pred_ptr[j + 1];
  for (int64_t p = p0; p < p1; ++p) {
    // budget test of Algorithm 1: opt[L, t] + c <= B, i.e. opt[L, t] <= tau
    const int32_t tau = Beff - pc[p];
    if (tau < 0) continue;                    // no source cell can pass
    const int32_t dt = pdt[p];
    const int32_t i = pidx[p];
    const int32_t wi = w[i];
    if (dt >= tile0 + kTile || dt + wi <= tile0) continue;  // window misses the tile
    const uint16_t* src = m + row_off[i];
    const uint32_t kadd = ((uint32_t)pdm[p] << 16) | (uint32_t)i;
#pragma unroll
    for (int r = 0; r < kCellsPerThread; r++) {
      const int32_t t = tile0 + r * kFillThreads + (int32_t)threadIdx.x - dt;
      if ((uint32_t)t < (uint32_t)wi) {
        const uint32_t x = src[t];
        if (x <= (uint32_t)tau) acc[r] = min(acc[r], (x << 16) + kadd);
      }
    }
  }
  uint16_t* mo = m + row_off[j];
  uint16_t* ao = arg + row_off[j];
#pragma unroll
  for (int r = 0; r < kCellsPerThread; r++) {
    const int32_t tp = tile0 + r * kFillThreads + (int32_t)threadIdx.x;
    if (tp < wj) {
      mo[tp] = (uint16_t)(acc[r] >> 16);
      ao[tp] = (uint16_t)(acc[r] & 0xFFFFu);
    }
  }
}

// t* = min (time-centric) or max (memory-centric) finite t of row V.
__global__ void k_select(const uint16_t* m, const int64_t* row_off, int64_t v, const int32_t* w,
                         int objective, DevStatus* st) {
  const int64_t off = row_off[v];
  const int32_t wv = w[v];
  for (int32_t t = blockIdx.x * blockDim.x + threadIdx.x; t < wv; t += gridDim.x * blockDim.x) {
    if (m[off + t] != kInfM) {
      if (objective == RC_TIME_CENTRIC)
        atomicMin(&st->t_sel, t);
      else
        atomicMax(&st->t_sel, t);
    }
  }
}

__global__ void k_select_finish(const uint16_t* m, const int64_t* row_off, int64_t v,
                                DevStatus* st) {
  if (threadIdx.x != 0) return;
  if (st->t_sel == INT32_MAX) st->t_sel = -1;
  st->m_sel = st->t_sel >= 0 ? (int32_t)m[row_off[v] + st->t_sel] : -1;
}

// Traceback of optarg from (V, t*) (Section 4.2), then Eq. 1 and Eq. 2 of
// the chain from their definitions: U_i is the union of boundaries of
// L_1..L_i, segment i needs M(U_{i-1}) + 2 M(V_i) + A(L_i), the overhead is
// T(V \ U_k).  One wave; lane w holds word w of the sets.
__global__ __launch_bounds__(kWave) void k_trace(
    int64_t F, int n, int words, int64_t fstride, const uint64_t* __restrict__ bits,
    const uint64_t* __restrict__ bd, const int32_t* __restrict__ Tsum,
    const int32_t* __restrict__ Msum, const int32_t* __restrict__ Tbd,
    const int32_t* __restrict__ A, const int32_t* __restrict__ T, const int32_t* __restrict__ M,
    const int32_t* __restrict__ w, const int64_t* __restrict__ row_off,
    const uint16_t* __restrict__ arg, int64_t T_total, DevStatus* st, int32_t* chain,
    int32_t* seg, uint8_t* cached) {
  const int lane = threadIdx.x;
  const bool active = lane < words;
  int64_t j = F - 1;
  int64_t t = st->t_sel;
  int32_t k = 0;
  bool bad = t < 0;
  while (j != 0 && !bad) {
    if (t < 0 || t >= w[j]) {
      bad = true;
      break;
    }
    const uint32_t a = arg[row_off[j] + t];
    if (a == kNoArg || a >= (uint32_t)j || k >= F) {
      bad = true;
      break;
    }
    const int64_t i = a;
    const uint64_t x = active ? bits[(int64_t)lane * fstride + i] & bd[(int64_t)lane * fstride + j] : 0ull;
    const int64_t ti = wave_sum_i64(active ? word_cost(x, lane, T) : 0);
    t -= (int64_t)Tsum[j] - Tbd[j] - Tsum[i] + ti;   // T((L_j \ L_i) \ bd(L_j))
    if (lane == 0) chain[k] = (int32_t)j;
    k++;
    j = i;
  }
  if (t != 0) bad = true;                             // the walk must end at (empty, 0)
  if (bad) {
    if (lane == 0) {
      st->error = 2;
      st->k = -1;
    }
    return;
  }
  __syncthreads();
  for (int c = lane; c < k / 2; c += kWave) {         // chain in increasing order
    const int32_t tmp = chain[c];
    chain[c] = chain[k - 1 - c];
    chain[k - 1 - c] = tmp;
  }
  __syncthreads();
  for (int v = lane; v < n; v += kWave) seg[v] = -1;
  __syncthreads();
  uint64_t U = 0, prev = 0;
  int64_t peak = 0;
  for (int c = 0; c < k; c++) {
    const int64_t s = chain[c];
    const uint64_t L = active ? bits[(int64_t)lane * fstride + s] : 0ull;
    const uint64_t Vi = L & ~prev;
    const int64_t mu = wave_sum_i64(active ? word_cost(U, lane, M) : 0);
    const int64_t mv = wave_sum_i64(active ? word_cost(Vi, lane, M) : 0);
    const int64_t mem = mu + 2 * mv + A[s];
    peak = mem > peak ? mem : peak;
    for (uint64_t b = Vi; b; b &= b - 1) seg[lane * 64 + __builtin_ctzll(b)] = c;
    if (active) U |= bd[(int64_t)lane * fstride + s];
    prev = L;
  }
  for (int b = 0; b < 64 && active; b++) {
    const int v = lane * 64 + b;
    if (v < n) cached[v] = (uint8_t)((U >> b) & 1ull);
  }
  const int64_t tu = wave_sum_i64(active ? word_cost(U, lane, T) : 0);
  const int64_t mu = wave_sum_i64(active ? word_cost(U, lane, M) : 0);
  if (lane == 0) {
    st->k = k;
    st->overhead = T_total - tu;
    st->peak = peak;
    st->cache_mem = mu;
  }
}

}  // namespace

hipError_t launch_solve_init(rc_solution sol, hipStream_t s) {
  rc_family f = sol->f;
  hipLaunchKernelGGL(k_solve_init, dim3(1), dim3(64), 0, s, sol->m, sol->arg, f->row_off,
                     sol->objective, sol->status);
  return hipGetLastError();
}

hipError_t launch_fill(rc_solution sol, hipStream_t s) {
  rc_family f = sol->f;
  const int64_t L = (int64_t)f->level_ptr.size() - 1;
  for (int64_t l = 1; l < L; l++) {            // level 0 is the empty set
    const int64_t lb = f->level_ptr[l], le = f->level_ptr[l + 1];
    const int64_t tiles = (f->level_maxw[l] + kTile - 1) / kTile;
    if (tiles <= 0 || le <= lb) continue;
    hipLaunchKernelGGL(k_fill_level, dim3((unsigned)tiles, (unsigned)(le - lb)),
                       dim3(kFillThreads), 0, s, lb, f->w, f->row_off, f->pred_ptr, f->pidx,
                       f->pdt, f->pdm, f->pc, (int32_t)sol->Beff, sol->m, sol->arg);
  }
  return hipGetLastError();
}

hipError_t launch_select(rc_solution sol, hipStream_t s) {
  rc_family f = sol->f;
  const int64_t v = f->F - 1;
  const int64_t wv = f->w_host[v];
  const unsigned blocks = (unsigned)std::min<int64_t>((wv + 255) / 256, 1024);
  hipLaunchKernelGGL(k_select, dim3(blocks > 0 ? blocks : 1), dim3(256), 0, s, sol->m, f->row_off,
                     v, f->w, sol->objective, sol->status);
  hipLaunchKernelGGL(k_select_finish, dim3(1), dim3(64), 0, s, sol->m, f->row_off, v,
                     sol->status);
  return hipGetLastError();
}

hipError_t launch_trace(rc_solution sol, hipStream_t s) {
  rc_family f = sol->f;
  rc_graph g = f->g;
  hipLaunchKernelGGL(k_trace, dim3(1), dim3(kWave), 0, s, f->F, g->n, g->words, f->fstride,
                     f->bits, f->bd, f->Tsum, f->Msum, f->Tbd, f->A, g->dT, g->dM, f->w,
                     f->row_off, sol->arg, g->T_total, sol->status, sol->chain, sol->seg, sol->cached);
  return hipGetLastError();
}

}  // namespace rcdp
