// Ghost-zone wavefront DP fill for wide tables (Algorithm 1, pull form).
//
// Geometry (as in blocked.hip).  Rows are stored right-aligned: row L ends
// on a 64-cell boundary E_L and the cell at distance u <= 0 from the row
// end (t = P_L + u, P_L = w_L - 1) sits at E_L - 1 + u.  A pair (L_i, L_j)
// with right-aligned shift e = T(bd(L_i) \ bd(L_j)) >= 0 relaxes target
// cell u from source cell u + e, so a cell only reads cells at the same or
// a smaller distance from the row end.  Column c owns the C cells
// u in [u0, u0 + C), u0 = -(c + 1) C + 1.
//
// Blocks.  Targets 1..F-1 (family order) are cut into blocks of at most kJB
// consecutive targets such that the dependency cone of the block stays
// within H = kGhostHalo cells: cone(r) = max over later rows r2 of the
// block with a pair (r, r2) of cone(r2) + e(r, r2), cone(last) = 0, and
// every cone(r) <= H (ghost_cut).  A column then computes the H cells to
// its right (the leftmost cells of column c - 1) as well, for every row of
// the block: row r is exact on u < u0 + C + H - cone(r), which covers what
// the later rows of the block read from it, so the block needs no cell of
// another column that is being computed at the same time.
//
// Schedule.  A workgroup takes the next column from an atomic ticket (right
// to left) and runs it through every block.  Per block:
//  - panel: every source before the block (all final) relaxes the C + H
//    cells of all rows of the block.  Records (one per source and cluster
//    of nearby shifts, blocks.hip) stream through a software pipeline:
//    headers and source windows are copied global -> LDS by DMA two stages
//    ahead.  Sources before the previous block come first; they only need
//    the columns to the right to have finished the block before the
//    previous one, which they almost always have.  Only then does the
//    column wait for the previous block in the columns its windows reach
//    (progress[c'] >= first row of this block).
//  - triangle: row by row, the row is final; it goes to an LDS buffer, its
//    own C cells are stored, and it relaxes the later rows of the block
//    from the buffer (shifts <= H).  One barrier per row; nothing waits for
//    another workgroup.
//  - publish: once the block's stores have completed, progress[c] = the
//    first row after the block.
// A column only waits for columns with smaller tickets, held by workgroups
// that are already running, so the fill progresses without relying on
// co-residency.  Every wait is bounded (timeout -> error flag, exit).
//
// Waves.  All five waves compute (lane l holds cells u0 + l + q * 320);
// waves 0-3 issue the panel DMA (two records each), so their memory counter
// holds nothing else while the pipeline runs, and wave 4 polls the
// progress of other columns.
//
// Coherence.  Every cell is written exactly once, by the column that owns
// it, with an agent-coherent store; readers load agent-coherently, and only
// rows that a column has published after its stores completed.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>

#include "ghost_cut.h"
#include "rc_internal.h"
#include "wavefront.h"

namespace rcdp {

namespace {

using namespace wf;

constexpr int kGW = 5;                   // waves per workgroup, all compute
constexpr int kGT = kGW * kWave;         // threads
constexpr int kDW = 4;                   // waves that issue the panel DMA
constexpr int kPoll = kGW - 1;           // wave that polls other columns

template <int CPT>
struct GGeo {
  static constexpr int CH = kGT * CPT;             // cells computed per column
  static constexpr int C = CH - kGhostHalo;        // cells owned per column
  static constexpr int WIN = CH + kSpan + 8;       // staged cells per record window
  static constexpr int NCH = WIN / 8;              // 16-byte chunks per window
  static constexpr int IPR = (NCH + 63) / 64;      // DMA instructions per window
  static constexpr int D = 2;                      // pipeline stages in flight
  static constexpr int NWB = D + 1;                // window buffers
  static constexpr int NHB = 2 * D + 1;            // header buffers
  static constexpr int NI = 2 * IPR + 1;           // DMA instructions per DMA wave per stage
  static constexpr int RBUF = CH + kGhostHalo + 8; // row buffer with an infinity tail
  static_assert(C % 64 == 0, "a column holds whole 128-byte lines");
  static_assert(WIN % 8 == 0 && kSpan + 8 <= 256, "panel window");
  static_assert(NI * (D - 1) < 63, "vmcnt range");
  static_assert(D < NWB && 2 * D < NHB, "buffer counters wrap at most once");
};

template <int CPT>
__global__ __launch_bounds__(kGT) void k_fill_ghost(GParams p0, const GParams* gps, int32_t nb) {
  using G = GGeo<CPT>;
  constexpr int CH = G::CH, C = G::C, D = G::D, NWB = G::NWB, NHB = G::NHB, NI = G::NI;
  constexpr int WIN = G::WIN, NCH = G::NCH, IPR = G::IPR, RBUF = G::RBUF;
  __shared__ __attribute__((aligned(16))) uint16_t s_win[NWB][kNB][WIN];
  __shared__ __attribute__((aligned(16))) int32_t s_hdr[NHB][kNB][kRecInts];
  __shared__ __attribute__((aligned(16))) uint16_t s_row[2][RBUF];
  __shared__ int32_t s_tk;
  __shared__ int32_t s_gate[2];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid & (kWave - 1);
  const bool dmaw = wave < kDW;
  const u16x2 kInf2 = (u16x2)((unsigned short)kInfM);
  for (int x = CH + tid; x < RBUF; x += kGT) {      // the tails read as infinity
    s_row[0][x] = (uint16_t)kInfM;
    s_row[1][x] = (uint16_t)kInfM;
  }
  auto bar = []() __attribute__((always_inline)) {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  };
  int32_t gate_seq = 0;                               // parity of the gate slots

  while (true) {
    if (tid == 0) s_tk = atomicAdd(p0.ticket, 1);
    bar();
    const int32_t tk = __builtin_amdgcn_readfirstlane(s_tk);
    bar();                                            // s_tk is read before it is rewritten
    if (tk >= p0.K * nb) return;
    const int32_t c = tk / nb;
    const GParams p = batch_params(p0, gps, nb, tk);
    gint32* const progress = (gint32*)p.progress;
    gstatus* const gst = (gstatus*)p.st;
    cint32* const meta = (cint32*)p.meta;
    cint32* const tri = (cint32*)p.tri;
    cint32* const bstart = (cint32*)p.bstart;
    cint64* const clu_ptr = (cint64*)p.clu_ptr;
    cint32* const live = (cint32*)p.live;
    const int32_t u0 = -(c + 1) * C + 1;              // u of the column's first cell
    const int64_t cC = (int64_t)c * C;
    const int32_t cl = c < p.cap ? c : p.cap - 1;

    // Wait until progress[c'] >= need for the columns c' in [c - reach, c):
    // wave kPoll polls, all waves meet at a barrier per poll.  False: timeout.
    auto gate = [&](int32_t need, int32_t reach) __attribute__((always_inline)) -> bool {
      reach = reach < c ? reach : c;
      const long long t0 = wall_clock64();
      while (true) {
        if (wave == kPoll) {
          bool ok = true;
          for (int32_t d0 = 1; d0 <= reach && ok; d0 += kWave) {
            const int32_t d = d0 + lane;
            ok = __all(d > reach || ld_relaxed(&progress[c - d]) >= need);
          }
          const int32_t res = ok ? 1 : (wall_clock64() - t0 > p.timeout_ticks ? -1 : 0);
          if (lane == 0) s_gate[gate_seq & 1] = res;
        }
        bar();
        const int32_t res = __builtin_amdgcn_readfirstlane(s_gate[gate_seq & 1]);
        ++gate_seq;
        if (res != 0) return res > 0;
      }
    };

    for (int32_t b = 0; b < p.nblk; ++b) {
      jitter_delay(p.jitter, c, b, tid / kWave);
      cint32* const mt = meta + (int64_t)b * kMetaInts;
      const int32_t s0 = bstart[b], s1 = bstart[b + 1];
      if (cC > mt[3]) {                              // no row of the block reaches the column
        if (tid == 0)
          __hip_atomic_store(&progress[c], s1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        continue;
      }
      const int32_t nrows = s1 - s0;
      cint32* const lv = live + ((int64_t)b * p.cap + cl) * 2;
      const int32_t nO = lv[0], nN = lv[1];          // live records of this column per group
      const int32_t nOall = mt[4];                   // the new group starts there
      const int32_t SO = (nO + kNB - 1) / kNB;
      const int32_t S = SO + (nN + kNB - 1) / kNB;   // pipeline stages
      const int32_t needO = b > 0 ? bstart[b - 1] : 1, needN = s0;
      const int32_t reachO = (kGhostHalo + mt[1] + C - 1) / C;
      const int32_t reachN = (kGhostHalo + mt[5] + C - 1) / C;
      const int32_t* const pcrec = p.crec + clu_ptr[b] * kRecInts;

      // record of stage k, slot kk (stages [0, SO) old group, then new)
      auto rec_of = [&](int32_t k, int kk, bool& valid) __attribute__((always_inline)) -> int32_t {
        if (k < SO) {
          const int32_t r = k * kNB + kk;
          valid = r < nO;
          return valid ? r : 0;
        }
        const int32_t r = (k - SO) * kNB + kk;
        valid = r < nN;
        return valid ? nOall + r : 0;
      };
      // stage k goes to window buffer wb = k % NWB and header buffer hb = k % NHB
      auto issue_hdr = [&](int32_t k, int hb) __attribute__((always_inline)) {
        if (dmaw && lane < 16) {
          bool valid;
          const int32_t r = rec_of(k, 2 * wave + (lane >> 3), valid);
          const int32_t* src = pcrec + (int64_t)r * kRecInts + (lane & 7) * 4;
          dma16(src, __builtin_amdgcn_readfirstlane(lds_addr(&s_hdr[hb][2 * wave][0])));
        }
      };
      auto issue_win = [&](int32_t k, int wb, int hb) __attribute__((always_inline)) {
        if (!dmaw) return;
#pragma unroll
        for (int h = 0; h < 2; h++) {
          const int kk = 2 * wave + h;
          bool valid;
          (void)rec_of(k, kk, valid);
          const WinDma wd = win_dma(s_hdr[hb][kk], valid, u0, CH, p.m);
#pragma unroll
          for (int i = 0; i < IPR; i++) {
            const int32_t kc = lane + 64 * i;
            if (kc < NCH) {
              const bool ok = kc >= wd.lo && kc < wd.hi;
              dma16(ok ? (const void*)(wd.base + 8 * kc) : (const void*)p.sentinel,
                    __builtin_amdgcn_readfirstlane(lds_addr(&s_win[wb][kk][512 * i])));
            }
          }
        }
      };
      // gate levels: stages of the old group need needO, the new group needN
      int32_t gated = 0;
      auto gate_for = [&](int32_t k) __attribute__((always_inline)) -> bool {
        const int32_t lvl = k < SO ? 1 : 2;
        if (gated < 1 && !gate(needO, reachO)) return false;
        if (lvl == 2 && gated < 2 && !gate(needN, reachN)) return false;
        gated = gated > lvl ? gated : lvl;
        return true;
      };

      auto run = [&](auto NP_) __attribute__((always_inline)) -> bool {
        constexpr int NP = decltype(NP_)::value;     // packed target pairs of the block
        u16x2 acc[NP][CPT];
#pragma unroll
        for (int x = 0; x < NP; x++)
#pragma unroll
          for (int q = 0; q < CPT; q++) acc[x][q] = kInf2;

        // ---------------- panel
        auto compute = [&](int wb, int hb) __attribute__((always_inline)) {
#pragma unroll
          for (int kk = 0; kk < kNB; kk++) {
            const int4* h4 = reinterpret_cast<const int4*>(s_hdr[hb][kk]);
            const int4 o0 = h4[2], o1 = h4[3], tt = h4[4], dd = h4[5];
            const int32_t off[kJB] = {o0.x, o0.y, o0.z, o0.w, o1.x, o1.y, o1.z, o1.w};
            const u16x2 tau[4] = {as_u16x2(tt.x), as_u16x2(tt.y), as_u16x2(tt.z), as_u16x2(tt.w)};
            const u16x2 dm[4] = {as_u16x2(dd.x), as_u16x2(dd.y), as_u16x2(dd.z), as_u16x2(dd.w)};
            const uint16_t* wk = &s_win[wb][kk][tid];
#pragma unroll
            for (int q = 0; q < CPT; q++)
#pragma unroll
              for (int pp = 0; pp < NP; pp++) {
                u16x2 x;
                x.x = wk[off[2 * pp] + q * kGT];
                x.y = wk[off[2 * pp + 1] + q * kGT];
                acc[pp][q] = relax2(acc[pp][q], x, tau[pp], dm[pp]);
              }
          }
        };
        if (S > 0) {
#pragma unroll
          for (int32_t k = 0; k < D; k++) issue_hdr(k, k % NHB);
          wait_vm<0>();
          bar();
          if (!gate_for(S < D ? S - 1 : D - 1)) return false;
#pragma unroll
          for (int32_t k = 0; k < D; k++) {
            issue_win(k, k % NWB, k % NHB);
            issue_hdr(k + D, (k + D) % NHB);
          }
          int wb = 0, hb = 0;                          // k % NWB, k % NHB
          for (int32_t k = 0; k < S; k++) {
            if (dmaw) {
              if (k + D <= S)
                wait_vm<NI*(D - 1)>();
              else
                wait_vm<0>();
            }
            bar();
            compute(wb, hb);
            if (k + D < S) {
              if (!gate_for(k + D)) return false;
              issue_win(k + D, wb + D >= NWB ? wb + D - NWB : wb + D,
                        hb + D >= NHB ? hb + D - NHB : hb + D);
              issue_hdr(k + 2 * D, hb + 2 * D >= NHB ? hb + 2 * D - NHB : hb + 2 * D);
            }
            wb = wb + 1 == NWB ? 0 : wb + 1;
            hb = hb + 1 == NHB ? 0 : hb + 1;
          }
        }

        // ---------------- triangle: rows of the block in order
        cint32* const tr = tri + (int64_t)b * kJB * kTriInts;
#pragma unroll
        for (int r = 0; r < 2 * NP; r++) {
          if (r >= nrows) break;
          cint32* const pd = tr + r * kTriInts;
          const int32_t Pj = pd[12];
          const int64_t endj = (int64_t)(uint32_t)pd[13] | ((int64_t)pd[14] << 32);
          uint16_t* const rb = s_row[r & 1];
#pragma unroll
          for (int q = 0; q < CPT; q++) {
            const int32_t u = u0 + q * kGT + tid;
            const uint16_t v = (r & 1) ? acc[r >> 1][q].y : acc[r >> 1][q].x;
            rb[q * kGT + tid] = (u >= -Pj && u <= 0) ? v : (uint16_t)kInfM;
          }
          bar();
          if ((int64_t)Pj >= cC) {                     // the row has cells in this column
            const int64_t E = endj + 1;
            const int64_t Sr = E - (int64_t)((Pj + kRowAlign) / kRowAlign) * kRowAlign;
            if (tid < C / 8) {
              const int64_t g = E - (int64_t)(c + 1) * C + 8 * tid;
              if (g >= Sr) st_sc1(p.m + g, *reinterpret_cast<const u32x4*>(&rb[8 * tid]));
            }
          }
#pragma unroll
          for (int pp = 0; pp < NP; pp++) {
            if (2 * pp + 1 <= r) continue;              // targets at or before row r
            const uint32_t o = (uint32_t)pd[pp];
            const int32_t o0 = (int32_t)(o & 0xFFFFu), o1 = (int32_t)(o >> 16);
            const u16x2 tau = as_u16x2(pd[4 + pp]), dm = as_u16x2(pd[8 + pp]);
#pragma unroll
            for (int q = 0; q < CPT; q++) {
              u16x2 x;
              x.x = rb[o0 + q * kGT + tid];
              x.y = rb[o1 + q * kGT + tid];
              acc[pp][q] = relax2(acc[pp][q], x, tau, dm);
            }
          }
        }
        // ---------------- publish: rows < s1 of this column are stored
        wait_vm<0>();
        bar();
        jitter_delay(p.jitter, c, b, 16);
        if (tid == 0)
          __hip_atomic_store(&progress[c], s1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return true;
      };

      bool ok;
      const int32_t np = (nrows + 1) / 2;
      if (np <= 1)
        ok = run(std::integral_constant<int, 1>{});
      else if (np == 2)
        ok = run(std::integral_constant<int, 2>{});
      else if (np == 3)
        ok = run(std::integral_constant<int, 3>{});
      else
        ok = run(std::integral_constant<int, 4>{});
      if (!ok) {
        wait_vm<0>();                                // no DMA may land after the exit
        if (tid == 0) gst->error = 3;
        return;
      }
    }
  }
}

// near[j * kNear + d - 1]: shift e of the pair (L_{j-d}, L_j), -1 without
// one.  Predecessor lists are sorted by ascending source, so the pairs with
// sources j - kNear .. j - 1 are the last entries of j's list.
__global__ void k_near_shifts(int64_t F, const int32_t* w, const int64_t* pred_ptr,
                              const int32_t* pidx, const int32_t* pdt, int32_t* near) {
  for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < F;
       j += (int64_t)gridDim.x * blockDim.x) {
    int32_t e[kNear];
#pragma unroll
    for (int d = 0; d < kNear; d++) e[d] = -1;
    for (int64_t q = pred_ptr[j + 1] - 1; q >= pred_ptr[j]; q--) {
      const int32_t i = pidx[q];
      const int64_t d = j - i;
      if (d > kNear) break;
      if (d >= 1) e[d - 1] = (w[j] - w[i]) - pdt[q];
    }
#pragma unroll
    for (int d = 0; d < kNear; d++) near[j * kNear + d] = e[d];
  }
}

// Per solve, the in-block lists of every block: for row r (target j0 + r)
// the later rows of the block as packed pairs of targets (2p, 2p + 1):
// [p] the two shifts (LDS offsets into the row buffer) as uint16, [4 + p]
// the budgets B - c, [8 + p] the additions dm (a dead target: 0, 0,
// 0xFFFF); [12] P_j, [13..14] index of the cell u = 0 of row j.  A live
// shift above the halo contradicts the cut and is reported as an error.
__global__ void k_ghost_tri(int64_t nblk, const int32_t* bstart, int32_t Beff, const int32_t* w,
                            const int64_t* row_off, BlockRecords R, int32_t* tri,
                            DevStatus* st) {
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < nblk * kJB;
       x += (int64_t)gridDim.x * blockDim.x) {
    const int64_t b = x / kJB;
    const int r = (int)(x % kJB);
    const int64_t j0 = bstart[b];
    const int64_t j = j0 + r;
    int32_t* d = tri + x * kTriInts;
    uint32_t off[kJB / 2] = {0, 0, 0, 0}, tau[kJB / 2] = {0, 0, 0, 0};
    uint32_t dm[kJB / 2] = {0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};
    int32_t Pj = -1;
    int64_t endj = 0;
    if (j < bstart[b + 1]) {
      Pj = w[j] - 1;
      endj = row_off[j] + Pj;
      for (int s2 = r + 1; s2 < kJB && j0 + s2 < bstart[b + 1]; s2++) {
        const int64_t t = b * kJB * kJB + (int64_t)r * kJB + s2;
        const int32_t e = R.tri_e[t];
        const int32_t tv = Beff - R.tri_c[t];
        if (e < 0 || tv < 0) continue;
        if (e > kGhostHalo) {
          st->error = 4;
          continue;
        }
        const int sh = 16 * (s2 & 1);
        off[s2 / 2] |= (uint32_t)e << sh;
        tau[s2 / 2] |= (uint32_t)tv << sh;
        dm[s2 / 2] = (dm[s2 / 2] & ~(0xFFFFu << sh)) | ((R.tri_kadd[t] >> 16) << sh);
      }
    }
    for (int p = 0; p < kJB / 2; p++) {
      d[p] = (int32_t)off[p];
      d[4 + p] = (int32_t)tau[p];
      d[8 + p] = (int32_t)dm[p];
    }
    d[12] = Pj;
    d[13] = (int32_t)(endj & 0xFFFFFFFF);
    d[14] = (int32_t)(endj >> 32);
    d[15] = 0;
  }
}

__global__ void k_ghost_init(int32_t* progress, int32_t K, int32_t* ticket) {
  for (int32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < K; k += gridDim.x * blockDim.x)
    progress[k] = 1;                        // the empty set's row is written by the init kernel
  if (blockIdx.x == 0 && threadIdx.x == 0) *ticket = 0;
}

template <int CPT>
hipError_t launch_cpt(const GParams& prm, const GParams* gps, int32_t nb, int32_t grid,
                      hipEvent_t e0, hipEvent_t e1, hipStream_t s) {
  if (e0 && hipEventRecord(e0, s) != hipSuccess) return hipErrorUnknown;
  hipLaunchKernelGGL(k_fill_ghost<CPT>, dim3(grid), dim3(kGT), 0, s, prm, gps, nb);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (e1 && hipEventRecord(e1, s) != hipSuccess) return hipErrorUnknown;
  return hipSuccess;
}

int64_t wait_ticks() {
  int dev = 0;
  int clock_khz = 0;
  (void)hipGetDevice(&dev);
  if (hipDeviceGetAttribute(&clock_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
      clock_khz <= 0)
    clock_khz = 100000;
  return (int64_t)clock_khz * 1000 * 4;                // 4 s per wait
}

int32_t cells_per_column(int cpt) { return kGT * cpt - kGhostHalo; }

// Per-table preparation (records, in-block lists) and the kernel parameters.
hipError_t prepare_table(rc_solution sol, int32_t C, int32_t K, int32_t* ticket, GParams* prm,
                         hipStream_t s) {
  rc_family f = sol->f;
  hipLaunchKernelGGL(k_ghost_init, dim3((K + 255) / 256), dim3(256), 0, s, sol->progress, K,
                     ticket);
  hipError_t pe = launch_pad_init(sol, s);
  if (pe == hipSuccess) pe = launch_rec_prepare(sol, s);
  if (pe == hipSuccess) pe = launch_rec_sort(sol, C, kGhostHalo, s);
  if (pe != hipSuccess) return pe;
  const int64_t nt = f->nblk * kJB;
  hipLaunchKernelGGL(k_ghost_tri, dim3((unsigned)std::min<int64_t>((nt + 255) / 256, 1024)),
                     dim3(256), 0, s, f->nblk, f->bstart, (int32_t)sol->Beff, f->w, f->row_off,
                     f->rec, sol->tri, sol->status);
  pe = hipGetLastError();
  if (pe != hipSuccess) return pe;
  prm->F = (int32_t)f->F;
  prm->nblk = (int32_t)f->nblk;
  prm->K = K;
  prm->bstart = f->bstart;
  prm->clu_ptr = f->clu_ptr;
  prm->crec = sol->crec;
  prm->meta = sol->blk_meta;
  prm->tri = sol->tri;
  prm->live = sol->live;
  prm->cap = sol->live_cap;
  prm->sentinel = sol->sentinel;
  prm->m = sol->m;
  prm->progress = sol->progress;
  prm->ticket = ticket;
  prm->st = sol->status;
  prm->timeout_ticks = wait_ticks();
  prm->jitter = jitter_seed();
  return hipSuccess;
}

hipError_t launch_kernel(const GParams& prm, const GParams* gps, int32_t nb, int cpt,
                         hipEvent_t e0, hipEvent_t e1, hipStream_t s) {
  // Any grid size is correct; more workgroups than columns would idle.
  const int64_t cols = (int64_t)prm.K * nb;
  const int32_t grid = (int32_t)std::min<int64_t>(cols, (int64_t)num_cus() * 4);
  if (std::getenv("RCDP_DEBUG"))
    std::fprintf(stderr, "rcdp: ghost fill %d table(s) x K=%d columns of %d cells, grid=%d\n", nb,
                 prm.K, cells_per_column(cpt), grid);
  if (cpt == 1) return launch_cpt<1>(prm, gps, nb, grid, e0, e1, s);
  return launch_cpt<2>(prm, gps, nb, grid, e0, e1, s);
}

}  // namespace

std::vector<int32_t> ghost_cut(int64_t F, const std::vector<int32_t>& near) {
  return ghost_cut_rows(F, near, kNear, kJB, kGhostHalo);
}

hipError_t launch_near_shifts(rc_family f, int32_t* near, hipStream_t s) {
  const unsigned grid = (unsigned)std::min<int64_t>((f->F + 255) / 256, 1024);
  hipLaunchKernelGGL(k_near_shifts, dim3(grid > 0 ? grid : 1), dim3(256), 0, s, f->F, f->w,
                     f->pred_ptr, f->pidx, f->pdt, near);
  return hipGetLastError();
}

// Two cells per thread (576-cell columns) once the table is wide enough to
// keep the CUs busy with them; RCDP_GHOST_CPT=1|2 overrides.
int ghost_cells_per_thread(rc_family f) {
  if (const char* env = std::getenv("RCDP_GHOST_CPT")) {
    const int v = std::atoi(env);
    if (v == 1 || v == 2) return v;
  }
  return (f->max_row + cells_per_column(2) - 1) / cells_per_column(2) >= 2 * num_cus() ? 2 : 1;
}

int64_t ghost_columns(rc_family f) {
  const int32_t C = cells_per_column(ghost_cells_per_thread(f));
  return (f->max_row + C - 1) / C;
}

hipError_t launch_fill_ghost(rc_solution sol, hipStream_t s) {
  rc_family f = sol->f;
  if (f->F < 2) return hipSuccess;
  const int cpt = ghost_cells_per_thread(f);
  const int32_t C = cells_per_column(cpt);
  const int32_t K = (int32_t)((f->max_row + C - 1) / C);
  GParams prm;
  const hipError_t pe = prepare_table(sol, C, K, sol->ticket, &prm, s);
  if (pe != hipSuccess) return pe;
  return launch_kernel(prm, nullptr, 1, cpt, sol->evk0, sol->evk1, s);
}

hipError_t launch_fill_ghost_batch(rc_solution* sols, int32_t nb, GParams* host_prm,
                                   GParams* dev_prm, hipStream_t s) {
  rc_family f = sols[0]->f;
  if (f->F < 2) return hipSuccess;
  const int cpt = ghost_cells_per_thread(f);
  const int32_t C = cells_per_column(cpt);
  const int32_t K = (int32_t)((f->max_row + C - 1) / C);
  for (int32_t b = 0; b < nb; b++) {
    // every table resets the shared ticket; they all run before the kernel
    const hipError_t pe = prepare_table(sols[b], C, K, sols[0]->ticket, &host_prm[b], s);
    if (pe != hipSuccess) return pe;
  }
  const hipError_t ce = hipMemcpyAsync(dev_prm, host_prm, sizeof(GParams) * (size_t)nb,
                                       hipMemcpyHostToDevice, s);
  if (ce != hipSuccess) return ce;
  return launch_kernel(host_prm[0], dev_prm, nb, cpt, sols[0]->evk0, sols[0]->evk1, s);
}

}  // namespace rcdp
