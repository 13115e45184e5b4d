// Blocked wavefront DP fill for wide tables.
//
// Geometry.  Rows are stored right-aligned: row L ends on a 64-cell
// boundary E_L, and the cell at distance u <= 0 from the row end
// (t = P_L + u, P_L = w_L - 1) sits at E_L - 1 + u.  Column c of every row
// holds u in [-(c+1)C + 1, -cC], i.e. whole 128-byte lines of one row.  A
// pair with right-aligned shift e (see blocks.hip) reads source cells
// u = u' + e for target cells u': column c reads the source row in
// columns c - ceil(e / C) .. c, never to the left of c.
//
// Schedule.  A workgroup takes the next column from an atomic ticket and
// runs it through every target block in family order; only afterwards
// does it take another column.  Columns are handed out right to left and
// a column only ever waits for columns with smaller tickets, held by
// workgroups that are already running, so the fill always progresses
// without relying on co-residency.  progress[c] counts the rows finished
// in column c (agent-scope release after each row; acquire after each
// wait).
//
// Work per block [j0, j1) of one column:
//  A. wait until the columns the panel reaches have finished rows < j0;
//     for each panel record (source i): stage the union of the block's
//     windows of row i in LDS once, then relax every target of the block
//     from it into registers (slots whose shift lies outside the staged
//     span read global memory directly);
//  B. for each target j of the block in order: store its column (final:
//     every predecessor of j has been applied), publish it, then stage row
//     j and push it to the later targets of the block that contain it.
// Each relaxation is Algorithm 1's update: the source value x passes the
// budget test iff x <= B - c, and the candidate key is ((x + dm) << 16) | i;
// the unsigned minimum keeps the smallest m' and, among equal m', the
// smallest source index, which is what the strict update of Algorithm 1
// over ascending sources keeps.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>

#include "rc_internal.h"

namespace rcdp {

namespace {

constexpr int kWave = 64;
constexpr int kBT = 256;                 // threads per workgroup

struct BParams {
  int64_t F;
  int64_t nblk;
  int32_t K;                             // columns
  int32_t Beff;
  const int32_t* w;
  const int64_t* row_off;
  const int64_t* rec_ptr;
  BlockRecords R;
  uint16_t* m;
  uint16_t* arg;
  int32_t* progress;
  int32_t* ticket;
  DevStatus* st;
  int64_t timeout_ticks;
};

__device__ __forceinline__ int32_t ld_relaxed(const int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wave 0 waits until progress[c - d] >= need for d = 1..reach (columns to
// the right).  Returns false when it gave up (timeout or abort flag).
__device__ bool wait_columns(const BParams& p, int32_t c, int32_t reach, int32_t need) {
  const int lane = threadIdx.x & (kWave - 1);
  if (reach > c) reach = c;
  for (int32_t d0 = 1; d0 <= reach; d0 += kWave) {
    const int32_t d = d0 + lane;
    bool ok = d > reach;
    const long long t0 = wall_clock64();
    while (true) {
      if (!ok) ok = ld_relaxed(&p.progress[c - d]) >= need;
      if (__all(ok)) break;
      if (wall_clock64() - t0 > p.timeout_ticks || ld_relaxed(&p.st->error) != 0) return false;
      __builtin_amdgcn_s_sleep(1);
    }
  }
  return true;
}

__device__ __forceinline__ void publish(const BParams& p, int32_t c, int32_t rows) {
  __hip_atomic_store(&p.progress[c], rows, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

template <int CPT>
__global__ __launch_bounds__(kBT) void k_fill_blocked(BParams p) {
  constexpr int C = kBT * CPT;           // cells per column
  constexpr int SPAN = C;                // shifts staged together: [emin, emin + SPAN]
  constexpr int WIN = C + SPAN;
  __shared__ uint16_t win[WIN];
  __shared__ int32_t s_col;
  __shared__ int32_t s_abort;
  const int tid = threadIdx.x;
  const int wave = tid / kWave;

  while (true) {
    if (tid == 0) {
      s_col = atomicAdd(p.ticket, 1);
      s_abort = 0;
    }
    __syncthreads();
    const int32_t c = s_col;
    if (c >= p.K) return;
    const int32_t u0 = -(c + 1) * C + 1;          // u of slot 0 of this column

    for (int64_t b = 0; b < p.nblk; ++b) {
      const int64_t j0 = 1 + b * kJB;
      const int64_t j1 = j0 + kJB < p.F ? j0 + kJB : p.F;
      int32_t maxP = -1;
      for (int64_t j = j0; j < j1; j++) maxP = max(maxP, p.w[j] - 1);
      if ((int64_t)c * C > maxP) {                 // no target of the block reaches here
        __syncthreads();
        if (tid == 0) publish(p, c, (int32_t)j1);
        continue;
      }
      // ---- A. panel: sources older than the block
      if (wave == 0) {
        const int32_t reach = (p.R.blk_emax[b] + C - 1) / C;
        if (!wait_columns(p, c, reach, (int32_t)j0)) {
          if ((tid & (kWave - 1)) == 0) {
            __hip_atomic_store(&p.st->error, 3, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_abort = 1;
          }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      }
      __syncthreads();
      if (s_abort) return;

      uint32_t acc[kJB][CPT];
#pragma unroll
      for (int s = 0; s < kJB; s++)
#pragma unroll
        for (int q = 0; q < CPT; q++) acc[s][q] = 0xFFFFFFFFu;

      for (int64_t r = p.rec_ptr[b]; r < p.rec_ptr[b + 1]; ++r) {
        const int32_t i = p.R.src[r];
        const int32_t emin = p.R.emin[r];
        const int32_t emax = p.R.emax[r];
        const int32_t Pi = p.w[i] - 1;
        const int64_t endi = p.row_off[i] + Pi;     // index of u = 0
        if (u0 + C - 1 + emax < -Pi) continue;      // every window lies before the row
        const int32_t span = min(emax - emin, SPAN);
        const uint16_t* srow = p.m + endi;
        for (int x = tid; x < C + span; x += kBT) {
          const int32_t u = u0 + emin + x;
          win[x] = (u >= -Pi && u <= 0) ? srow[u] : (uint16_t)kInfM;
        }
        __syncthreads();
#pragma unroll
        for (int s = 0; s < kJB; s++) {
          const int32_t e = p.R.e[r * kJB + s];
          const int32_t tau = p.Beff - p.R.c[r * kJB + s];
          if (e < 0 || tau < 0) continue;
          const uint32_t kadd = p.R.kadd[r * kJB + s];
          const int32_t off = e - emin;
          if (off <= span) {
#pragma unroll
            for (int q = 0; q < CPT; q++) {
              const uint32_t x = win[q * kBT + tid + off];
              if (x <= (uint32_t)tau) acc[s][q] = min(acc[s][q], (x << 16) + kadd);
            }
          } else {
#pragma unroll
            for (int q = 0; q < CPT; q++) {
              const int32_t u = u0 + q * kBT + tid + e;
              if (u >= -Pi && u <= 0) {
                const uint32_t x = srow[u];
                if (x <= (uint32_t)tau) acc[s][q] = min(acc[s][q], (x << 16) + kadd);
              }
            }
          }
        }
        __syncthreads();
      }

      // ---- B. targets of the block in order: store, publish, push
#pragma unroll
      for (int s = 0; s < kJB; s++) {
        const int64_t j = j0 + s;
        if (j < j1) {
          const int32_t Pj = p.w[j] - 1;
          const int64_t endj = p.row_off[j] + Pj;
#pragma unroll
          for (int q = 0; q < CPT; q++) {
            const int32_t up = u0 + q * kBT + tid;
            if (up >= -Pj) {
              p.m[endj + up] = (uint16_t)(acc[s][q] >> 16);
              p.arg[endj + up] = (uint16_t)(acc[s][q] & 0xFFFFu);
            }
          }
          __syncthreads();
          if (tid == 0) publish(p, c, (int32_t)(j + 1));
          const int32_t temax = p.R.tri_emax[b * kJB + s];
          if (s + 1 < kJB && temax >= 0) {
            if (wave == 0) {
              const int32_t reach = (temax + C - 1) / C;
              if (!wait_columns(p, c, reach, (int32_t)(j + 1))) {
                if ((tid & (kWave - 1)) == 0) {
                  __hip_atomic_store(&p.st->error, 3, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                  s_abort = 1;
                }
              }
              __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            }
            __syncthreads();
            if (s_abort) return;
            const int32_t span = min(temax, SPAN);
            const uint16_t* srow = p.m + endj;
            for (int x = tid; x < C + span; x += kBT) {
              const int32_t u = u0 + x;
              win[x] = (u >= -Pj && u <= 0) ? srow[u] : (uint16_t)kInfM;
            }
            __syncthreads();
#pragma unroll
            for (int s2 = s + 1; s2 < kJB; s2++) {
              const int64_t t = b * kJB * kJB + (int64_t)s * kJB + s2;
              const int32_t e = p.R.tri_e[t];
              const int32_t tau = p.Beff - p.R.tri_c[t];
              if (e < 0 || tau < 0) continue;
              const uint32_t kadd = p.R.tri_kadd[t];
              if (e <= span) {
#pragma unroll
                for (int q = 0; q < CPT; q++) {
                  const uint32_t x = win[q * kBT + tid + e];
                  if (x <= (uint32_t)tau) acc[s2][q] = min(acc[s2][q], (x << 16) + kadd);
                }
              } else {
#pragma unroll
                for (int q = 0; q < CPT; q++) {
                  const int32_t u = u0 + q * kBT + tid + e;
                  if (u >= -Pj && u <= 0) {
                    const uint32_t x = srow[u];
                    if (x <= (uint32_t)tau) acc[s2][q] = min(acc[s2][q], (x << 16) + kadd);
                  }
                }
              }
            }
            __syncthreads();
          }
        }
      }
    }
  }
}

__global__ void k_blocked_init(int32_t* progress, int32_t K, int32_t* ticket) {
  for (int32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < K; k += gridDim.x * blockDim.x)
    progress[k] = 1;                        // the empty set's row is written by the init kernel
  if (blockIdx.x == 0 && threadIdx.x == 0) *ticket = 0;
}

template <int CPT>
hipError_t launch_cpt(const BParams& prm, int32_t grid, hipStream_t s) {
  hipLaunchKernelGGL(k_fill_blocked<CPT>, dim3(grid), dim3(kBT), 0, s, prm);
  return hipGetLastError();
}

int g_num_cus = -1;

}  // namespace

// Column width: cells per lane in 1..4 (256..1024 cells); the choice
// minimises the per-CU share of columns times the column width, preferring
// wider columns (more reuse of staged windows) on ties.
int blocked_cells_per_thread(rc_family f) {
  if (g_num_cus < 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&g_num_cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      g_num_cus = 256;
  }
  const char* env = std::getenv("RCDP_CPT");
  if (env && env[0] >= '1' && env[0] <= '4') return env[0] - '0';
  int best = 4;
  int64_t best_cost = INT64_MAX;
  for (int cpt = 4; cpt >= 1; cpt--) {
    const int64_t C = (int64_t)kBT * cpt;
    const int64_t K = (f->max_row + C - 1) / C;
    const int64_t cost = (K + g_num_cus - 1) / g_num_cus * C;
    if (cost < best_cost) {
      best_cost = cost;
      best = cpt;
    }
  }
  return best;
}

int64_t blocked_columns(rc_family f) {
  const int64_t C = (int64_t)kBT * blocked_cells_per_thread(f);
  return (f->max_row + C - 1) / C;
}

hipError_t launch_fill_blocked(rc_solution sol, hipStream_t s) {
  rc_family f = sol->f;
  if (f->F < 2) return hipSuccess;
  const int cpt = blocked_cells_per_thread(f);
  const int32_t K = (int32_t)((f->max_row + (int64_t)kBT * cpt - 1) / ((int64_t)kBT * cpt));
  int dev = 0;
  int clock_khz = 0;
  (void)hipGetDevice(&dev);
  if (hipDeviceGetAttribute(&clock_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
      clock_khz <= 0)
    clock_khz = 100000;
  hipLaunchKernelGGL(k_blocked_init, dim3((K + 255) / 256), dim3(256), 0, s, sol->progress, K,
                     sol->ticket);
  BParams prm;
  prm.F = f->F;
  prm.nblk = f->nblk;
  prm.K = K;
  prm.Beff = (int32_t)sol->Beff;
  prm.w = f->w;
  prm.row_off = f->row_off;
  prm.rec_ptr = f->rec_ptr;
  prm.R = f->rec;
  prm.m = sol->m;
  prm.arg = sol->arg;
  prm.progress = sol->progress;
  prm.ticket = sol->ticket;
  prm.st = sol->status;
  prm.timeout_ticks = (int64_t)clock_khz * 1000 * 4;   // 4 s per wait
  // Any grid size is correct; more workgroups than columns would idle.
  const int32_t grid = (int32_t)std::min<int64_t>(K, (int64_t)g_num_cus * 4);
  if (std::getenv("RCDP_DEBUG"))
    std::fprintf(stderr, "rcdp: blocked fill K=%d columns of %d cells, grid=%d, %lld blocks\n", K,
                 kBT * cpt, grid, (long long)f->nblk);
  switch (cpt) {
    case 1: return launch_cpt<1>(prm, grid, s);
    case 2: return launch_cpt<2>(prm, grid, s);
    case 3: return launch_cpt<3>(prm, grid, s);
    default: return launch_cpt<4>(prm, grid, s);
  }
}

}  // namespace rcdp
