// Blocked wavefront DP fill for wide tables (Algorithm 1, pull form).
//
// Geometry.  Rows are stored right-aligned: row L ends on a 64-cell
// boundary E_L, and the cell at distance u <= 0 from the row end
// (t = P_L + u, P_L = w_L - 1) sits at E_L - 1 + u.  Column c of every row
// holds u in [-(c+1)C + 1, -cC], whole 128-byte lines of one row.  A pair
// with right-aligned shift e (blocks.hip) relaxes target cell u from source
// cell u + e, so column c only reads columns c, c - 1, ... (to the right).
//
// Schedule.  A workgroup takes the next column from an atomic ticket and
// runs it through every block of kJB consecutive targets in family order.
// Columns are handed out right to left and a column only ever waits for
// columns with smaller tickets, held by workgroups that are already
// running, so the fill progresses without relying on co-residency.
//
// Work per block b of a column (targets j0 .. j0 + 7):
//  - the accumulators of the block already hold every source before the
//    block: the panel of older sources was applied while block b - 1 was
//    being finished, and the rows of block b - 1 pushed themselves;
//  - row by row: the row is final, so it is stored; then it pushes itself
//    to the later rows of the block and to every row of block b + 1, reading
//    its own cells of this column (in LDS), its halo (the cells to the right,
//    for shifts up to kHalo) and, for larger shifts, a window of its own;
//  - meanwhile the panel of block b + 1 (sources before block b, all final)
//    streams through a software pipeline: record headers and source windows
//    are copied global -> LDS by DMA several stages ahead of the relaxation.
//
// Waves.  Four compute waves own the cells (CPT per lane) and issue only
// the pipeline's DMA, so their memory counter holds nothing else and the
// pipeline waits for exactly the stage it needs.  A fifth, control wave
// stores finished rows, stages halos and windows, and polls other
// columns.  All five meet once per step at a barrier; control state travels
// through LDS slots alternating by step parity, so a slot is never written
// in the step in which it is read.
//
// Coherence.  Every table cell is written exactly once, by the column that
// owns it, with an agent-coherent store (sc1); before the fill every cell
// holds kPendM.  Halo and window loads read agent-coherently and poll: a
// chunk that still holds kPendM is loaded again.  The panel reads whole rows
// of blocks that are finished; a column publishes how many rows it has
// finished (progress[c]) once its stores have completed, and the panel
// waits for the columns it reaches.
//
// Relaxation.  m' = x + dm if x <= tau (tau = B - c), else infinity, for two
// targets at once in packed unsigned 16-bit lanes with saturation:
// y = x +sat dm, q = x -sat tau is nonzero exactly when the budget test
// fails, and q * 0xFFFF +sat y (one multiply-add with clamp) is then 0xFFFF,
// else y.  All finite values stay below kPendM, so the saturated value is
// the infinity code.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>

#include "rc_internal.h"
#include "wavefront.h"

namespace rcdp {

namespace {

using namespace wf;

constexpr int kCW = 4;                   // compute waves
constexpr int kBT = kCW * kWave;         // compute threads
constexpr int kThreads = kBT + kWave;    // plus the control wave
constexpr uint32_t kUnset = 0xFFFD;      // LDS cell whose staging load has not landed

template <int CPT>
struct Geo {
  static constexpr int C = kBT * CPT;              // cells per column
  static constexpr int WIN = C + 256;              // staged cells per panel record
  static constexpr int NCH = WIN / 8;              // 16-byte chunks per record window
  static constexpr int IPR = (NCH + 63) / 64;      // DMA instructions per record window
  static constexpr int D = 2;                      // pipeline stages in flight
  static constexpr int NW = D + 1;                 // window buffers
  static constexpr int NH = 2 * D + 1;             // header buffers
  static constexpr int NI = 2 * IPR + 1;           // DMA instructions per compute wave per stage
  static constexpr int RB = C + kHalo + 8;         // row buffer: own cells + halo
  static constexpr int FB = C + 8;                 // far window
  static constexpr int NCF = FB / 8;               // chunks per far window
  static constexpr int PUSH = 2 * RB + kFarMax * FB;
  static constexpr int CPL = C / kWave;            // cells per control lane when storing a row
  static_assert(kSpan + 7 <= 256, "panel window");
  static_assert(NI * (D - 1) < 63, "vmcnt range");
  static_assert(D < NW && 2 * D < NH, "buffer counters wrap at most once");
};



// Does a chunk of 8 staged cells hold kUnset (not landed) / kPendM?
__device__ __forceinline__ bool has_half(u32x4 v, uint32_t code) {
  bool r = false;
#pragma unroll
  for (int x = 0; x < 4; x++) r |= (v[x] & 0xFFFFu) == code || (v[x] >> 16) == code;
  return r;
}

// One launch fills nb tables of the same family (different budgets): the
// ticket t takes column t / nb of table t % nb, so every table's columns are
// still handed out right to left and a column only waits for columns with
// smaller tickets.  nb = 1: the table of p0; else bps[0 .. nb) (device).
template <int CPT>
__global__ __launch_bounds__(kThreads) void k_fill_blocked(BParams p0, const BParams* bps,
                                                           int32_t nb) {
  using G = Geo<CPT>;
  constexpr int C = G::C, D = G::D, NW = G::NW, NH = G::NH, NI = G::NI, WIN = G::WIN;
  constexpr int NCH = G::NCH, IPR = G::IPR, RB = G::RB, FB = G::FB, NCF = G::NCF, CPL = G::CPL;
  __shared__ __attribute__((aligned(16))) uint16_t s_win[NW][kNB][WIN];
  __shared__ __attribute__((aligned(16))) int32_t s_hdr[NH][kNB][kRecInts];
  __shared__ __attribute__((aligned(16))) uint16_t s_push[G::PUSH];
  // control -> all, by step parity: {rows ready, abort, panel grant, -}; s_cur
  // is the control's current state, copied into the next step's slot
  __shared__ int32_t s_ctl[2][4];
  __shared__ int32_t s_cur[4];
  __shared__ int32_t s_col;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);   // wave-uniform
  const int lane = tid & (kWave - 1);
  const bool ctl = wave == kCW;
  // every step waits for the control wave's share of it while the compute
  // waves keep the SIMDs busy: let the control wave issue first
  if (ctl) __builtin_amdgcn_s_setprio(3);
  const u16x2 kInf2 = (u16x2)((unsigned short)kInfM);
  uint32_t step = 0;

  auto bar = [&]() __attribute__((always_inline)) {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    ++step;
  };
  auto ctl_write = [&]() __attribute__((always_inline)) {
    if (ctl && lane == 0) {
      s_ctl[(step + 1) & 1][0] = s_cur[0];
      s_ctl[(step + 1) & 1][1] = s_cur[1];
      s_ctl[(step + 1) & 1][2] = s_cur[2];
    }
  };
  auto cur_set = [&](int i, int32_t v) __attribute__((always_inline)) {
    if (lane == 0) s_cur[i] = v;
  };

  while (true) {
    if (ctl && lane == 0) {
      s_col = atomicAdd(p0.ticket, 1);
      s_cur[0] = -1;
      s_cur[1] = 0;
      s_cur[2] = 1;                                  // the panel of block 0 may start
    }
    ctl_write();
    bar();
    const int32_t tk = __builtin_amdgcn_readfirstlane(s_col);
    if (tk >= p0.K * nb) return;
    const int32_t c = tk / nb;
    const BParams p = batch_params(p0, bps, nb, tk);
    gint32* const progress = (gint32*)p.progress;
    gstatus* const gst = (gstatus*)p.st;
    cint32* const meta = (cint32*)p.meta;
    cint32* const push = (cint32*)p.push;
    cint64* const clu_ptr = (cint64*)p.clu_ptr;
    cint32* const live = (cint32*)p.live;
    ctl_write();                                   // the state the first step reads
    const int32_t u0 = -(c + 1) * C + 1;          // u of the column's first cell
    const int64_t cC = (int64_t)c * C;
    const int32_t cl = c < p.cap ? c : p.cap - 1;

    u16x2 acc[kJB / 2][CPT], nxt[kJB / 2][CPT];
#pragma unroll
    for (int x = 0; x < kJB / 2; x++)
#pragma unroll
      for (int q = 0; q < CPT; q++) nxt[x][q] = kInf2;

    // ---------------- panel pipeline (state identical in every wave).  The
    // panel of block pb runs as stages of kNB records: first the uniform
    // records live in this column (pnU, stages [0, pSU)), then the others
    // (pnG, from record pnu on).  It starts once the control grants it
    // (grant > pb), requests the first headers, then their windows, then
    // computes one stage per step.
    int32_t pb = -1, pn = 0, pns = 0, pSU = 0, pnU = 0, pnG = 0, pnu = 0, pphase = 0;
    int32_t pw = 0, ph = 0;                        // pn % NW and pn % NH, kept as counters
    const int32_t* pcrec = p.crec;
    int32_t poll_reach = 0, poll_need = 0;         // control: what the grant waits for
    long long poll_t0 = 0;

    auto rec_of = [&](int32_t k, int kk, bool& valid) __attribute__((always_inline)) -> int32_t {
      if (k < pSU) {
        const int32_t r = k * kNB + kk;
        valid = r < pnU;
        return valid ? r : 0;
      }
      const int32_t r = (k - pSU) * kNB + kk;
      valid = r < pnG;
      return valid ? pnu + r : 0;
    };
    // stage k goes to window buffer wb = k % NW and header buffer hb = k % NH
    auto issue_hdr = [&](int32_t k, int hb) __attribute__((always_inline)) {   // compute waves
      if (lane < 16) {
        bool valid;
        const int32_t r = rec_of(k, 2 * wave + (lane >> 3), valid);
        const int32_t* src = pcrec + (int64_t)r * kRecInts + (lane & 7) * 4;
        dma16(src, __builtin_amdgcn_readfirstlane(lds_addr(&s_hdr[hb][2 * wave][0])));
      }
    };
    auto issue_win = [&](int32_t k, int wb, int hb) __attribute__((always_inline)) {
#pragma unroll
      for (int h = 0; h < 2; h++) {
        const int kk = 2 * wave + h;
        bool valid;
        (void)rec_of(k, kk, valid);
        const WinDma wd = win_dma(s_hdr[hb][kk], valid, u0, C, p.m);
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
    // Relax every slot of the kNB records of stage k into nxt.  No branch
    // per record: a record past the list or whose window misses the source
    // row was staged from the infinity sentinel, so its candidates are
    // infinite.
    auto compute = [&](int32_t k, int wb, int hb) __attribute__((always_inline)) {
      if (k < pSU) {                     // every slot of these records has one shift
#pragma unroll
        for (int kk = 0; kk < kNB; kk++) {
          const int4* h4 = reinterpret_cast<const int4*>(s_hdr[hb][kk]);
          const int32_t a = s_hdr[hb][kk][7];
          const int4 tt = h4[4], dd = h4[5];
          const u16x2 tau[4] = {as_u16x2(tt.x), as_u16x2(tt.y), as_u16x2(tt.z), as_u16x2(tt.w)};
          const u16x2 dm[4] = {as_u16x2(dd.x), as_u16x2(dd.y), as_u16x2(dd.z), as_u16x2(dd.w)};
          const uint16_t* wk = &s_win[wb][kk][a + tid];
#pragma unroll
          for (int q = 0; q < CPT; q++) {
            const u16x2 x = (u16x2)(wk[q * kBT]);
#pragma unroll
            for (int pp = 0; pp < 4; pp++) nxt[pp][q] = relax2(nxt[pp][q], x, tau[pp], dm[pp]);
          }
        }
        return;
      }
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
          for (int pp = 0; pp < 4; pp++) {
            u16x2 x;
            x.x = wk[off[2 * pp] + q * kBT];
            x.y = wk[off[2 * pp + 1] + q * kBT];
            nxt[pp][q] = relax2(nxt[pp][q], x, tau[pp], dm[pp]);
          }
      }
    };
    // Plan the panel of block b1 (no memory traffic yet).  Its sources, the
    // rows before block b1 - 1, must be final in every column it reaches:
    // progress >= need in columns c - reach .. c.
    auto pipe_setup = [&](int32_t b1, int32_t need) __attribute__((always_inline)) {
      pb = b1;
      pn = 0;
      pw = 0;
      ph = 0;
      pns = 0;
      pphase = 0;
      if (b1 >= p.nblk) return;
      cint32* mt = meta + (int64_t)b1 * kMetaInts;
      if (cC > mt[3]) return;                        // no cell of block b1 in this column
      cint32* lv = live + ((int64_t)b1 * p.cap + cl) * 2;
      pnU = lv[0];
      pnG = lv[1];
      pnu = mt[4];
      pSU = (pnU + kNB - 1) / kNB;
      pns = pSU + (pnG + kNB - 1) / kNB;
      pcrec = p.crec + clu_ptr[b1] * kRecInts;
      poll_reach = (mt[1] + C - 1) / C;
      if (poll_reach > c) poll_reach = c;
      poll_need = need;
      poll_t0 = wall_clock64();
    };
    // the pipeline state is the same in every lane: keep it in scalars
    auto uniform = [&]() __attribute__((always_inline)) {
      pn = __builtin_amdgcn_readfirstlane(pn);
      pw = __builtin_amdgcn_readfirstlane(pw);
      ph = __builtin_amdgcn_readfirstlane(ph);
      pns = __builtin_amdgcn_readfirstlane(pns);
      pphase = __builtin_amdgcn_readfirstlane(pphase);
      pSU = __builtin_amdgcn_readfirstlane(pSU);
      pnU = __builtin_amdgcn_readfirstlane(pnU);
      pnG = __builtin_amdgcn_readfirstlane(pnG);
      pnu = __builtin_amdgcn_readfirstlane(pnu);
      pb = __builtin_amdgcn_readfirstlane(pb);
    };
    auto step_pre = [&]() __attribute__((always_inline)) {
      uniform();
      if (!ctl && pn < pns) {
        if (pphase == 1) {
          wait_vm<0>();
        } else if (pphase == 2) {
          if (pn + D <= pns)
            wait_vm<NI*(D - 1)>();
          else
            wait_vm<0>();
        }
      }
    };
    auto step_post = [&](int32_t grant) __attribute__((always_inline)) {
      uniform();
      if (pn < pns) {
        if (pphase == 2) {
          if (!ctl) {
            compute(pn, pw, ph);
            if (pn + D < pns) {
              const int pwD = pw + D >= NW ? pw + D - NW : pw + D;
              const int phD = ph + D >= NH ? ph + D - NH : ph + D;
              const int ph2D = ph + 2 * D >= NH ? ph + 2 * D - NH : ph + 2 * D;
              issue_win(pn + D, pwD, phD);
              issue_hdr(pn + 2 * D, ph2D);
            }
          }
          ++pn;
          pw = pw + 1 == NW ? 0 : pw + 1;
          ph = ph + 1 == NH ? 0 : ph + 1;
        } else if (pphase == 1) {
          if (!ctl)
            for (int32_t k = 0; k < D; k++) {
              issue_win(k, k % NW, k % NH);
              issue_hdr(k + D, (k + D) % NH);
            }
          pphase = 2;
        } else if (grant > pb) {
          if (!ctl)
            for (int32_t k = 0; k < D; k++) issue_hdr(k, k % NH);
          pphase = 1;
        }
      }
    };
    // control: grant the planned panel once the columns it reaches are far
    // enough (one poll per step)
    auto panel_poll = [&]() __attribute__((always_inline)) {
      if (pn >= pns || s_cur[2] > pb) return;
      bool ok = true;
      for (int32_t d0 = 0; d0 <= poll_reach && ok; d0 += kWave) {
        const int32_t d = d0 + lane;
        ok = __all(d > poll_reach || ld_relaxed(&progress[c - d]) >= poll_need);
      }
      if (ok)
        cur_set(2, pb + 1);
      else if (wall_clock64() - poll_t0 > p.timeout_ticks)
        cur_set(1, 1);
    };
    // One step: pipeline wait, barrier, control state, pipeline stage, the
    // control's work.  False: the fill was aborted.
    int32_t rr = -1;
    auto run_step = [&](auto&& ctl_work) __attribute__((always_inline)) -> bool {
      step_pre();
      bar();
      rr = s_ctl[step & 1][0];
      const bool go_on = s_ctl[step & 1][1] == 0;
      const int32_t grant = s_ctl[step & 1][2];
      if (!go_on) return false;
      step_post(grant);
      if (ctl) {
        ctl_work();
        panel_poll();
        ctl_write();
      }
      return true;
    };
    auto no_work = []() {};
    auto fail = [&]() {
      wait_vm<0>();                                // no DMA may land after the exit
      if (ctl && lane == 0) gst->error = 3;
    };

    // ---------------- the panel of block 0 (source: the empty set's row)
    pipe_setup(0, 1);
    while (pn < pns)
      if (!run_step(no_work)) return fail();
#pragma unroll
    for (int x = 0; x < kJB / 2; x++)
#pragma unroll
      for (int q = 0; q < CPT; q++) {
        acc[x][q] = nxt[x][q];
        nxt[x][q] = kInf2;
      }

    for (int32_t b = 0; b < p.nblk; ++b) {
      jitter_delay(p.jitter, c, b, threadIdx.x / kWave);
      const int64_t j0 = 1 + (int64_t)b * kJB;
      const int32_t nrows = meta[(int64_t)b * kMetaInts + 2];
      // the panel of block b + 1: rows before block b, final once the
      // columns it reaches have finished block b - 1
      pipe_setup(b + 1, (int32_t)j0);

      // rows of the block: final -> stored; pushed to later rows and block b + 1
      auto do_row = [&](auto S_) __attribute__((always_inline)) -> bool {
        constexpr int s = decltype(S_)::value;
        if (s >= nrows) return true;
        cint32* pd = push + ((int64_t)b * kJB + s) * kPushInts;
        const int32_t hs = pd[0], nfar = pd[1], maxPt = pd[2], emax = pd[3], Pj = pd[4];
        const int64_t endj = (int64_t)(uint32_t)pd[5] | ((int64_t)pd[6] << 32);
        const bool need = maxPt >= cC && (int64_t)Pj + emax >= cC;
        if (!need && cC > Pj) return true;           // no cell here and nothing to push
        const bool staged = need && (hs > 0 || nfar > 0);
        const int rb = (s & 1) * RB;
        const int64_t E = endj + 1;
        const int64_t S = E - (int64_t)((Pj + kRowAlign) / kRowAlign) * kRowAlign;
        if (!ctl) {                                  // finalize row s into its buffer
#pragma unroll
          for (int q = 0; q < CPT; q++) {
            const int32_t u = u0 + q * kBT + tid;
            const uint16_t v = (s & 1) ? acc[s >> 1][q].y : acc[s >> 1][q].x;
            s_push[rb + q * kBT + tid] = u >= -Pj ? v : (uint16_t)kInfM;
          }
        }
        long long t0 = 0;
        // reload the staged chunks that read a cell not written yet; report
        // the row ready when all have landed
        auto inspect_now = [&]() __attribute__((always_inline)) {
          bool unset = false;
          const int nh = hs / 8;
          if (lane < nh) {
            u32x4* ch = reinterpret_cast<u32x4*>(&s_push[rb + C + 8 * lane]);
            const u32x4 v = *ch;
            const bool out = has_half(v, kUnset);
            unset |= out;
            if (!out && has_half(v, kPendM)) {
              *ch = (u32x4)(kUnset | (kUnset << 16));
              wait_lds();
              dma16(p.m + (E - cC + 8 * lane), __builtin_amdgcn_readfirstlane(lds_addr(&s_push[rb + C])));
              unset = true;
            }
          }
          for (int k = 0; k < nfar; k++) {
            const int32_t e = pd[8 + k];
            const int64_t astart = endj + u0 + e - (e & 7);
#pragma unroll
            for (int i = 0; i < (NCF + 63) / 64; i++) {
              const int kc = lane + 64 * i;
              if (kc < NCF) {
                u32x4* ch = reinterpret_cast<u32x4*>(&s_push[2 * RB + k * FB + 8 * kc]);
                const u32x4 v = *ch;
                const bool out = has_half(v, kUnset);
                unset |= out;
                if (!out && has_half(v, kPendM)) {
                  *ch = (u32x4)(kUnset | (kUnset << 16));
                  wait_lds();
                  dma16(p.m + (astart + 8 * (int64_t)kc),
                        __builtin_amdgcn_readfirstlane(lds_addr(&s_push[2 * RB + k * FB + 512 * i])));
                  unset = true;
                }
              }
            }
          }
          if (!__any(unset))
            cur_set(0, s);
          else if (wall_clock64() - t0 > p.timeout_ticks)
            cur_set(1, 1);
        };
        // first step: the control stores the row and starts staging its reads
        auto store_and_stage = [&]() __attribute__((always_inline)) {
          const int64_t g = E - (int64_t)(c + 1) * C + (int64_t)CPL * lane;
          if (g >= S) {                              // whole lines inside the row
            const uint16_t* src = &s_push[rb + CPL * lane];
            if constexpr (CPL == 4) {
              st_sc1(p.m + g, *reinterpret_cast<const u32x2*>(src));
            } else {
#pragma unroll
              for (int x = 0; x < CPL / 8; x++)
                st_sc1(p.m + g + 8 * x, *reinterpret_cast<const u32x4*>(src + 8 * x));
            }
          }
          if (staged) {
            // halo: cells [u0 + C, u0 + C + hs) of row j, after the row's own
            // cells; one window per far target
            const u32x4 unset = (u32x4)(kUnset | (kUnset << 16));
            const int nh = hs / 8;
            if (lane < nh) *reinterpret_cast<u32x4*>(&s_push[rb + C + 8 * lane]) = unset;
            for (int k = 0; k < nfar; k++)
              for (int kc = lane; kc < NCF; kc += kWave)
                *reinterpret_cast<u32x4*>(&s_push[2 * RB + k * FB + 8 * kc]) = unset;
            wait_lds();
            if (lane < nh) {
              const int64_t gh = E - cC + 8 * lane;
              const bool ok = gh >= S && gh + 8 <= E;
              dma16(ok ? (const void*)(p.m + gh) : (const void*)p.sentinel,
                    __builtin_amdgcn_readfirstlane(lds_addr(&s_push[rb + C])));
            }
            for (int k = 0; k < nfar; k++) {
              const int32_t e = pd[8 + k];
              const int64_t astart = endj + u0 + e - (e & 7);
#pragma unroll
              for (int i = 0; i < (NCF + 63) / 64; i++) {
                const int kc = lane + 64 * i;
                if (kc < NCF) {
                  const int64_t gf = astart + 8 * (int64_t)kc;
                  const bool ok = gf >= S && gf + 8 <= E;
                  dma16(ok ? (const void*)(p.m + gf) : (const void*)p.sentinel,
                        __builtin_amdgcn_readfirstlane(
                            lds_addr(&s_push[2 * RB + k * FB + 512 * i])));
                }
              }
            }
          }
          if (staged) t0 = wall_clock64();
        };
        // later steps: inspect the staged chunks until the row is ready
        auto inspect = [&]() __attribute__((always_inline)) {
          if (rr >= s) return;
          inspect_now();
        };
        if (!run_step(store_and_stage)) return false;
        if (staged)
          while (true) {
            if (!run_step(inspect)) return false;
            if (rr >= s) break;
          }
        if (!ctl && need) {                          // push row s
          int32_t offs[kJB], taus[kJB], dms[kJB];
#pragma unroll
          for (int x = 0; x < kJB; x++) {
            offs[x] = pd[24 + x];
            taus[x] = pd[32 + x];
            dms[x] = pd[40 + x];
          }
#pragma unroll
          for (int pp = 0; pp < kJB; pp++) {
            if (pp < kJB / 2 && 2 * pp + 1 <= s) continue;   // targets before or at s
            int32_t o0 = offs[pp] & 0xFFFF, o1 = (int32_t)((uint32_t)offs[pp] >> 16);
            o0 += o0 < RB ? rb : 0;
            o1 += o1 < RB ? rb : 0;
            const u16x2 tau = as_u16x2(taus[pp]), dm = as_u16x2(dms[pp]);
#pragma unroll
            for (int q = 0; q < CPT; q++) {
              u16x2 x;
              x.x = s_push[o0 + q * kBT + tid];
              x.y = s_push[o1 + q * kBT + tid];
              if (pp < kJB / 2)
                acc[pp][q] = relax2(acc[pp][q], x, tau, dm);
              else
                nxt[pp - kJB / 2][q] = relax2(nxt[pp - kJB / 2][q], x, tau, dm);
            }
          }
        }
        return true;
      };
      if (!do_row(std::integral_constant<int, 0>{}) || !do_row(std::integral_constant<int, 1>{}) ||
          !do_row(std::integral_constant<int, 2>{}) || !do_row(std::integral_constant<int, 3>{}) ||
          !do_row(std::integral_constant<int, 4>{}) || !do_row(std::integral_constant<int, 5>{}) ||
          !do_row(std::integral_constant<int, 6>{}) || !do_row(std::integral_constant<int, 7>{}))
        return fail();

      // rest of the panel of block b + 1
      while (pn < pns)
        if (!run_step(no_work)) return fail();
      // publish: rows < j0 + nrows of this column are stored
      auto publish = [&]() __attribute__((always_inline)) {
        wait_vm<0>();
        jitter_delay(p.jitter, c, b, 16);
        if (lane == 0)
          __hip_atomic_store(&progress[c], (int32_t)(j0 + nrows), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
        cur_set(0, -1);
      };
      if (!run_step(publish)) return fail();
#pragma unroll
      for (int x = 0; x < kJB / 2; x++)
#pragma unroll
        for (int q = 0; q < CPT; q++) {
          acc[x][q] = nxt[x][q];
          nxt[x][q] = kInf2;
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
hipError_t launch_cpt(const BParams& prm, const BParams* bps, int32_t nb, int32_t grid,
                      hipEvent_t e0, hipEvent_t e1, hipStream_t s) {
  if (e0 && hipEventRecord(e0, s) != hipSuccess) return hipErrorUnknown;
  hipLaunchKernelGGL(k_fill_blocked<CPT>, dim3(grid), dim3(kThreads), 0, s, prm, bps, nb);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (e1 && hipEventRecord(e1, s) != hipSuccess) return hipErrorUnknown;
  return hipSuccess;
}

}  // namespace

int num_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] <= 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        v <= 0)
      v = 256;
    cached[dev] = v;
  }
  return cached[dev];
}

// Column width: 256, 512 or 1024 cells (1, 2 or 4 cells per compute lane).
// A column's time is dominated by its sequence of steps (one per panel stage
// or row handshake), which barely depends on the width, so the narrowest
// columns spread the table over the most workgroups; only very wide tables
// (more columns than about eight workgroups per CU could take) use wider
// columns.
int blocked_cells_per_thread(rc_family f) {
  const char* env = std::getenv("RCDP_CPT");
  if (env && (env[0] == '1' || env[0] == '2' || env[0] == '4')) return env[0] - '0';
  const int64_t k1 = (f->max_row + kBT - 1) / kBT;
  return k1 <= 8 * (int64_t)num_cus() ? 1 : 4;
}

int64_t blocked_columns(rc_family f) {
  const int64_t C = (int64_t)kBT * blocked_cells_per_thread(f);
  return (f->max_row + C - 1) / C;
}

namespace {

int64_t wait_ticks() {
  int dev = 0;
  int clock_khz = 0;
  (void)hipGetDevice(&dev);
  if (hipDeviceGetAttribute(&clock_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
      clock_khz <= 0)
    clock_khz = 100000;
  return (int64_t)clock_khz * 1000 * 4;                // 4 s per wait
}

// Per-table preparation (records, push lists, pending marks) and the kernel
// parameters of that table.
hipError_t prepare_table(rc_solution sol, int32_t C, int32_t K, int32_t* ticket, BParams* prm,
                         hipStream_t s) {
  rc_family f = sol->f;
  hipLaunchKernelGGL(k_blocked_init, dim3((K + 255) / 256), dim3(256), 0, s, sol->progress, K,
                     ticket);
  hipError_t pe = launch_fill_pending(sol, s);
  if (pe == hipSuccess) pe = launch_pad_init(sol, s);
  if (pe == hipSuccess) pe = launch_rec_prepare(sol, s);
  if (pe == hipSuccess) pe = launch_rec_sort(sol, C, 0, s);
  if (pe == hipSuccess) pe = launch_push_prepare(sol, C, s);
  if (pe != hipSuccess) return pe;
  prm->F = (int32_t)f->F;
  prm->nblk = (int32_t)f->nblk;
  prm->K = K;
  prm->w = f->w;
  prm->row_off = f->row_off;
  prm->clu_ptr = f->clu_ptr;
  prm->crec = sol->crec;
  prm->meta = sol->blk_meta;
  prm->push = sol->push;
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

hipError_t launch_kernel(const BParams& prm, const BParams* bps, int32_t nb, int cpt,
                         hipEvent_t e0, hipEvent_t e1, hipStream_t s) {
  // Any grid size is correct; more workgroups than columns would idle.
  const int64_t cols = (int64_t)prm.K * nb;
  const int32_t grid = (int32_t)std::min<int64_t>(cols, (int64_t)num_cus() * 4);
  if (std::getenv("RCDP_DEBUG"))
    std::fprintf(stderr, "rcdp: blocked fill %d table(s) x K=%d columns of %d cells, grid=%d\n",
                 nb, prm.K, kBT * cpt, grid);
  if (cpt == 1) return launch_cpt<1>(prm, bps, nb, grid, e0, e1, s);
  if (cpt == 2) return launch_cpt<2>(prm, bps, nb, grid, e0, e1, s);
  return launch_cpt<4>(prm, bps, nb, grid, e0, e1, s);
}

}  // namespace

hipError_t launch_fill_blocked(rc_solution sol, hipStream_t s) {
  rc_family f = sol->f;
  if (f->F < 2) return hipSuccess;
  const int cpt = blocked_cells_per_thread(f);
  const int32_t C = kBT * cpt;
  const int32_t K = (int32_t)((f->max_row + C - 1) / C);
  BParams prm;
  const hipError_t pe = prepare_table(sol, C, K, sol->ticket, &prm, s);
  if (pe != hipSuccess) return pe;
  return launch_kernel(prm, nullptr, 1, cpt, sol->evk0, sol->evk1, s);
}

hipError_t launch_fill_blocked_batch(rc_solution* sols, int32_t nb, BParams* host_prm,
                                     BParams* dev_prm, hipStream_t s) {
  rc_family f = sols[0]->f;
  if (f->F < 2) return hipSuccess;
  const int cpt = blocked_cells_per_thread(f);
  const int32_t C = kBT * cpt;
  const int32_t K = (int32_t)((f->max_row + C - 1) / C);
  for (int32_t b = 0; b < nb; b++) {
    // every table resets the shared ticket; they all run before the kernel
    const hipError_t pe = prepare_table(sols[b], C, K, sols[0]->ticket, &host_prm[b], s);
    if (pe != hipSuccess) return pe;
  }
  const hipError_t ce = hipMemcpyAsync(dev_prm, host_prm, sizeof(BParams) * (size_t)nb,
                                       hipMemcpyHostToDevice, s);
  if (ce != hipSuccess) return ce;
  return launch_kernel(host_prm[0], dev_prm, nb, cpt, sols[0]->evk0, sols[0]->evk1, s);
}

}  // namespace rcdp
