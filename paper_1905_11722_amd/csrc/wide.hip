// Wavefront DP fill for wide tables with split panel waves (Algorithm 1,
// pull form).
//
// Geometry (shared with the other wavefront fills).  Rows are stored
// right-aligned: the cell at distance u <= 0 from the end of row L (t = P_L + u,
// P_L = w_L - 1) sits at end_L + u, and at least kGuard infinite cells
// separate consecutive rows (and follow the last one).  Column c of every row
// holds u in [u0, u0 + kWC), u0 = -(c+1) kWC + 1.  A pair (L_i, L_j) with
// right-aligned shift e = T(bd(L_i) \ bd(L_j)) >= 0 relaxes target cell u from
// source cell u + e, so column c only reads columns c, c - 1, ... (to its
// right).  Columns are handed out right to left from an atomic ticket; a
// column only waits for columns with smaller tickets, which are already
// running, so the fill needs no co-residency.
//
// Targets 1..F-1 come in blocks of kJB.  For block b of a column:
//  - panel(b): the contributions of every source before the previous block
//    (rows < j0(b-1)), one record per (block, source, shift): the source row's
//    window of kWC cells at shift e and, per target slot, the budget term
//    tau = B - c and the addition dm;
//  - pushes: each row of block b-1 relaxes the rows of block b, and each row
//    of block b the later rows of its own block, once it is final.
//
// Waves.  Wave 0 (the row wave) owns the accumulators of the current block
// and finishes its rows one by one: store, then push into the later rows of
// the block and into the next block, reading its own cells from LDS and the
// cells of the columns to its right (written by other workgroups) from the
// table, polling until they hold no kPendM.  Waves 1..NP (panel waves) stream
// the panel of the next block meanwhile, every wave over all kWC cells of the
// column (4 cells per lane) and a disjoint share of the records, with no
// barrier: a record's budgets, additions and window base arrive in scalar
// registers, its window is four 2-byte loads per lane, and 64 packed VALU
// instructions relax its 2048 cells.  At the end of the block the panel waves'
// partial minima meet in LDS and become the next block's accumulators (two
// barriers per block); the column then publishes its progress.
//
// Coherence.  Every cell is written once, with an agent-coherent store, by
// the column that owns it; before the fill every cell holds kPendM.  The
// panel reads rows that every column it reaches has published (progress[c]
// counts the rows finished in column c, stored after the column's stores
// have completed), through agent-coherent loads.  The row wave reads other
// columns' cells of rows not yet published and repeats a load that returns
// kPendM.  Every wait is bounded (timeout -> abort -> RC_E_DEVICE).
//
// Relaxation.  m' = x + dm if x <= tau, else infinity, for two targets at once
// in packed unsigned 16-bit lanes with saturation (wavefront.h relax2).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <type_traits>

#include "rc_internal.h"
#include "wavefront.h"

namespace rcdp {

namespace {

using namespace wf;

constexpr uint32_t kBufFlags = 0x00020000u;   // raw buffer resource word 3 (gfx9)
constexpr int kSC1 = 16;                      // buffer load / store: agent-coherent (sc1)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0,
                                           (int)std::min<int64_t>(bytes, INT32_MAX), kBufFlags);
}

__device__ __forceinline__ uint16_t ld_cell(__amdgpu_buffer_rsrc_t r, int32_t voff, int32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, kSC1);
}

// A panel wave's partial minima: pair p = targets (2p, 2p+1), cell k = lane
// + 64 k of the column.
struct Acc {
  u16x2 v[kJB / 2][4];
};

__device__ __forceinline__ void acc_fill(Acc& a, u16x2 x) {
#pragma unroll
  for (int p = 0; p < kJB / 2; p++)
#pragma unroll
    for (int k = 0; k < 4; k++) a.v[p][k] = x;
}

// ---------------------------------------------------------------- panel
// The records of block pb that reach column c are [rb, rb + n) of the sorted
// list; panel wave pw (0..NP-1) takes records pw, pw + NP, ...  A record is
// its budgets and additions (8 words) and its window base and limit (2
// words), read by every lane of the wave (a broadcast load), and its window,
// four 2-byte loads per lane.  Software pipeline over the records of the
// wave: the budgets of record t + 1, the base of record t + 3 and the window
// of record t + 2 are issued, in that order, before record t is relaxed.
// The loads are compiler builtins, so the compiler counts them and waits
// for exactly what each instruction reads.
struct Td {
  u16x2 tau[kJB / 2], dm[kJB / 2];
};

__device__ __forceinline__ Td load_td(__amdgpu_buffer_rsrc_t rt, int32_t r) {
  typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
  const int32_t o = r * kWTd * 4;
  const i32x4 a = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(rt, 0, o, 0));
  const i32x4 d = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(rt, 0, o + 16, 0));
  Td t;
  t.tau[0] = as_u16x2(a.x);
  t.tau[1] = as_u16x2(a.y);
  t.tau[2] = as_u16x2(a.z);
  t.tau[3] = as_u16x2(a.w);
  t.dm[0] = as_u16x2(d.x);
  t.dm[1] = as_u16x2(d.y);
  t.dm[2] = as_u16x2(d.z);
  t.dm[3] = as_u16x2(d.w);
  return t;
}

__device__ __forceinline__ int2 load_bl(__amdgpu_buffer_rsrc_t rl, int32_t r) {
  typedef int32_t i32x2 __attribute__((ext_vector_type(2)));
  const i32x2 v = __builtin_bit_cast(i32x2, __builtin_amdgcn_raw_buffer_load_b64(rl, 0, r * 8, 0));
  return make_int2(v.x, v.y);
}

// The window of a record (its 4 cells per lane): the record's base moved to
// column c, clamped to its row's trailing guard (a window right of the row
// reads infinity there), or the table's trailing guard past the records.
__device__ __forceinline__ void load_window(__amdgpu_buffer_rsrc_t rm, int32_t null_off, int2 bl,
                                            bool live, int32_t cC2, int32_t voff,
                                            uint32_t (&x)[4]) {
  const int32_t o = voff + (live ? min(bl.x - cC2, bl.y) : null_off);
#pragma unroll
  for (int k = 0; k < 4; k++) x[k] = ld_cell(rm, o + 128 * k, 0);
}

// Each cell is kept in its own register (the load's low half): packing two
// cells into one register would wait for both loads at once.
__device__ __forceinline__ void relax_record(const Td& t, const uint32_t (&x)[4], Acc& nx) {
#pragma unroll
  for (int k = 0; k < 4; k++) {
    const u16x2 xw = __builtin_bit_cast(u16x2, x[k]);
    const u16x2 xx = xw.xx;                          // the cell (the load's low half), twice
#pragma unroll
    for (int q = 0; q < kJB / 2; q++) nx.v[q][k] = relax2(nx.v[q][k], xx, t.tau[q], t.dm[q]);
  }
}

template <int NP>
__device__ __forceinline__ void panel_records(const WParams& p, int32_t pw, int64_t rb, int32_t n,
                                              int32_t cC2, Acc& nx) {
  if (pw >= n) return;
  const __amdgpu_buffer_rsrc_t rm = rsrc(p.m, p.m_bytes);
  const __amdgpu_buffer_rsrc_t rt =
      rsrc(p.td + rb * kWTd, (int64_t)(p.rec_cap + kWPad - rb) * kWTd * 4);
  const __amdgpu_buffer_rsrc_t rl = rsrc(p.bl + rb * 2, (int64_t)(p.rec_cap + kWPad - rb) * 8);
  const int32_t voff = 2 * (int32_t)(threadIdx.x & (kWave - 1));
  // rings of three: slot j holds record r with (r - pw) / NP = j mod 3, so the
  // loop unrolled three times moves no register
  uint32_t x[3][4];
  Td t[3];
  int2 b[3];
  t[0] = load_td(rt, pw);
  b[0] = load_bl(rl, pw);
  b[1] = load_bl(rl, pw + NP);
  b[2] = load_bl(rl, pw + 2 * NP);
  load_window(rm, p.null_off, b[0], true, cC2, voff, x[0]);
  load_window(rm, p.null_off, b[1], pw + NP < n, cC2, voff, x[1]);
  // whole rounds of three records; a record past the end relaxes the
  // trailing guard's infinity (its budgets and base are never used)
  const int32_t rounds = ((n - pw + NP - 1) / NP + 2) / 3;
  int32_t r = pw;
  auto step = [&](auto J) __attribute__((always_inline)) {
    constexpr int j = decltype(J)::value;
    t[(j + 1) % 3] = load_td(rt, r + NP);
    b[j] = load_bl(rl, r + 3 * NP);
    asm volatile("" ::: "memory");   // keep the issue order: budgets, base, then the window
    load_window(rm, p.null_off, b[(j + 2) % 3], r + 2 * NP < n, cC2, voff, x[(j + 2) % 3]);
    relax_record(t[j], x[j], nx);
    r += NP;
  };
  for (int32_t it = 0; it < rounds; it++) {
    step(std::integral_constant<int, 0>{});
    step(std::integral_constant<int, 1>{});
    step(std::integral_constant<int, 2>{});
  }
}

// Is every column in [c - reach, c - 1] at least `need` rows far?  Polls until
// it is; false on timeout.
__device__ __forceinline__ bool gate(const WParams& p, int32_t c, int32_t reach, int32_t need) {
  const int lane = threadIdx.x & (kWave - 1);
  gint32* const progress = (gint32*)p.progress;
  const int32_t hi = min(reach, c);
  const long long t0 = wall_clock64();
  for (int32_t d0 = 1; d0 <= hi; d0 += kWave) {
    const int32_t d = d0 + lane;
    while (!__all(d > hi || ld_relaxed(&progress[c - d]) >= need)) {
      if (wall_clock64() - t0 > p.timeout_ticks) return false;
      __builtin_amdgcn_s_sleep(1);
    }
  }
  return true;
}

// ---------------------------------------------------------------- rows
// The row wave's accumulators live in LDS: acc[q][cell] holds targets
// (2q, 2q+1) of the current block, nxt[q][cell] its pushes into the next
// block, both as uint16 pairs, cell = lane + 64 k; row holds the row's own
// cells, then its halo.
struct RowLds {
  uint32_t acc[kJB / 2][kWC];
  uint32_t nxt[kJB / 2][kWC];
  uint16_t row[kWC + kWH + 8];
};

__device__ __forceinline__ int32_t lane_word(int32_t v, int i) {
  return __builtin_amdgcn_readlane(v, i);
}

// A row's push list, one word per lane (kWPush = 64 words).
__device__ __forceinline__ int32_t load_push(const WParams& p, int b, int s) {
  const int lane = threadIdx.x & (kWave - 1);
  const __amdgpu_buffer_rsrc_t rp = rsrc(p.push, (int64_t)p.nblk * kJB * kWPush * 4);
  return (int32_t)__builtin_amdgcn_raw_buffer_load_b32(
      rp, 4 * lane, (int32_t)(((int64_t)b * kJB + s) * kWPush * 4), 0);
}

// Cells of row j (end index endj, P = Pj) at u = ubase + lane + 64 k into
// out[k]; a cell outside [-Pj, 0] reads the trailing guard's infinity.  The
// loads go out together; loads that return kPendM (a cell of another column
// not written yet) are repeated.  False on timeout.
template <int N>
__device__ __forceinline__ bool load_row_cells(const WParams& p, __amdgpu_buffer_rsrc_t rm,
                                               int64_t endj, int32_t Pj, int32_t ubase,
                                               int nk, uint32_t (&out)[N]) {
  const int lane = threadIdx.x & (kWave - 1);
  if (ubase > 0 || ubase + 64 * nk - 1 < -Pj) {      // every cell lies outside the row
#pragma unroll
    for (int k = 0; k < N; k++) out[k] = kInfM;
    return true;
  }
  int32_t off[N];
#pragma unroll
  for (int k = 0; k < N; k++) {
    const int32_t u = ubase + lane + 64 * k;
    off[k] = (u <= 0 && u >= -Pj) ? (int32_t)(2 * (endj + u)) : p.null_off;
    if (k < nk) out[k] = ld_cell(rm, off[k], 0);
  }
  bool pend = false;
#pragma unroll
  for (int k = 0; k < N; k++) pend |= k < nk && out[k] == kPendM;
  if (!__any(pend)) return true;
  const long long t0 = wall_clock64();
  while (true) {
    __builtin_amdgcn_s_sleep(1);
    pend = false;
#pragma unroll
    for (int k = 0; k < N; k++)
      if (k < nk && out[k] == kPendM) {
        out[k] = ld_cell(rm, off[k], 0);
        pend |= out[k] == kPendM;
      }
    if (!__any(pend)) return true;
    if (wall_clock64() - t0 > p.timeout_ticks) return false;
  }
}

// Relax slot pair q (accumulators of the block or of the next one) with the
// source cells x[k] of the lane's four cells: the four accumulators are read
// before any is written, so that the pair waits for LDS once.
__device__ __forceinline__ void push_pair4(RowLds& L, int q, const u16x2 (&x)[4], u16x2 tau,
                                           u16x2 dm) {
  const int lane = threadIdx.x & (kWave - 1);
  uint32_t* a = q < kJB / 2 ? &L.acc[q][lane] : &L.nxt[q - kJB / 2][lane];
  uint32_t v[4];
#pragma unroll
  for (int k = 0; k < 4; k++) v[k] = a[64 * k];
#pragma unroll
  for (int k = 0; k < 4; k++)
    a[64 * k] = __builtin_bit_cast(uint32_t, relax2(__builtin_bit_cast(u16x2, v[k]), x[k], tau, dm));
}

// Issues the loads of the row's cells at u = ubase + lane + 64 k (k < 4);
// cells outside the row read the trailing guard's infinity.
__device__ __forceinline__ void far_loads(const WParams& p, __amdgpu_buffer_rsrc_t rm, int64_t endj,
                                          int32_t Pj, int32_t ubase, int32_t (&off)[4],
                                          uint32_t (&out)[4]) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int k = 0; k < 4; k++) {
    const int32_t u = ubase + lane + 64 * k;
    off[k] = (u <= 0 && u >= -Pj) ? (int32_t)(2 * (endj + u)) : p.null_off;
    out[k] = ld_cell(rm, off[k], 0);
  }
}

// Repeats the loads at byte offsets off[] that returned kPendM (not written
// yet) until none does; false on timeout.
template <int N>
__device__ __forceinline__ bool poll_cells(const WParams& p, __amdgpu_buffer_rsrc_t rm,
                                           const int32_t (&off)[N], uint32_t (&out)[N]) {
  bool pend = false;
#pragma unroll
  for (int k = 0; k < N; k++) pend |= out[k] == kPendM;
  if (!__any(pend)) return true;
  const long long t0 = wall_clock64();
  while (true) {
    __builtin_amdgcn_s_sleep(1);
    pend = false;
#pragma unroll
    for (int k = 0; k < N; k++)
      if (out[k] == kPendM) {
        out[k] = ld_cell(rm, off[k], 0);
        pend |= out[k] == kPendM;
      }
    if (!__any(pend)) return true;
    if (wall_clock64() - t0 > p.timeout_ticks) return false;
  }
}

// The far push of slot t (one slot of pair t / 2) with source cells f.
__device__ __forceinline__ void far_push(RowLds& L, int32_t pdv, int t, const uint32_t (&f)[4]) {
  const int q = t >> 1;
  const u16x2 tau = as_u16x2(lane_word(pdv, kWpTau + q)), dm = as_u16x2(lane_word(pdv, kWpDm + q));
  u16x2 x[4];
#pragma unroll
  for (int k = 0; k < 4; k++) {
    x[k].x = (t & 1) ? (uint16_t)kInfM : (uint16_t)f[k];
    x[k].y = (t & 1) ? (uint16_t)f[k] : (uint16_t)kInfM;
  }
  push_pair4(L, q, x, tau, dm);
}

// Row s of block b (push list pdv): store it, then push it into the later
// rows of the block (L.acc) and the rows of the next block (L.nxt).  False on
// timeout.
__device__ __forceinline__ bool row_step(const WParams& p, int32_t c, int s, int32_t pdv,
                                         RowLds& L) {
  const int lane = threadIdx.x & (kWave - 1);
  const int32_t Pj = lane_word(pdv, kWpP);
  const int64_t endj =
      (int64_t)(uint32_t)lane_word(pdv, kWpEnd) | ((int64_t)lane_word(pdv, kWpEnd + 1) << 32);
  const int32_t emax = lane_word(pdv, kWpEmax), maxPt = lane_word(pdv, kWpMaxPt);
  const int32_t cC = c * kWC;
  const int32_t u0 = -cC - kWC + 1;
  const bool need = maxPt >= cC && Pj + emax >= cC;   // a push reaches a cell of this column
  if (!need && cC > Pj) return true;                  // no cell here and nothing to push
  const __amdgpu_buffer_rsrc_t rm = rsrc(p.m, p.m_bytes);
  // the row is final: its cells of this column, infinity left of the row; a
  // store outside the row goes to an offset past the buffer and is dropped
  const uint16_t* accs = reinterpret_cast<const uint16_t*>(&L.acc[s >> 1][0]) + (s & 1);
  uint16_t v[4];
#pragma unroll
  for (int k = 0; k < 4; k++) {
    const int32_t u = u0 + lane + 64 * k;
    const uint16_t a = accs[2 * (lane + 64 * k)];
    v[k] = u >= -Pj ? a : (uint16_t)kInfM;
    __builtin_amdgcn_raw_buffer_store_b16(v[k], rm, u >= -Pj ? (int32_t)(2 * (endj + u)) : -1, 0,
                                          kSC1);
  }
  if (!need) return true;
  // own cells and the halo (cells of the columns to the right) in LDS
  const int32_t hs = lane_word(pdv, kWpHalo);
  const uint32_t far = (uint32_t)lane_word(pdv, kWpFar);
#pragma unroll
  for (int k = 0; k < 4; k++) L.row[lane + 64 * k] = v[k];
  if (hs > 0) {
    uint32_t h[kWH / 64];
    if (!load_row_cells<kWH / 64>(p, rm, endj, Pj, u0 + kWC, hs / 64, h)) return false;
#pragma unroll
    for (int k = 0; k < kWH / 64; k++)
      if (64 * k < hs) L.row[kWC + lane + 64 * k] = (uint16_t)h[k];
  }
  // near pushes: both slots of a pair from the row buffer (far slots read
  // infinity here and are relaxed below)
  uint32_t near_pairs = (uint32_t)lane_word(pdv, kWpNear);
  while (near_pairs) {
    const int q = __builtin_ctz(near_pairs);
    near_pairs &= near_pairs - 1;
    const int32_t e0 = lane_word(pdv, kWpE + 2 * q), e1 = lane_word(pdv, kWpE + 2 * q + 1);
    const bool n0 = e0 >= 0 && e0 <= kWH, n1 = e1 >= 0 && e1 <= kWH;
    const int32_t o0 = n0 ? e0 : 0, o1 = n1 ? e1 : 0;     // every read in range, used or not
    const u16x2 tau = as_u16x2(lane_word(pdv, kWpTau + q)), dm = as_u16x2(lane_word(pdv, kWpDm + q));
    uint16_t r0[4], r1[4];
#pragma unroll
    for (int k = 0; k < 4; k++) {
      r0[k] = L.row[lane + 64 * k + o0];
      r1[k] = L.row[lane + 64 * k + o1];
    }
    u16x2 x[4];
#pragma unroll
    for (int k = 0; k < 4; k++) {
      x[k].x = n0 ? r0[k] : (uint16_t)kInfM;
      x[k].y = n1 ? r1[k] : (uint16_t)kInfM;
    }
    push_pair4(L, q, x, tau, dm);
  }
  // far pushes (shift beyond the halo): the source cells straight from the
  // table, two slots at a time, both slots' loads in flight together (with
  // one slot left, the second is the same slot again: its push repeats the
  // first's values)
  uint32_t fm = far;
  while (fm) {
    const int ta = __builtin_ctz(fm);
    fm &= fm - 1;
    const int tb = fm ? __builtin_ctz(fm) : ta;
    fm &= fm - 1;
    int32_t oa[4], ob[4];
    uint32_t fa[4], fb[4];
    far_loads(p, rm, endj, Pj, u0 + lane_word(pdv, kWpE + ta), oa, fa);
    far_loads(p, rm, endj, Pj, u0 + lane_word(pdv, kWpE + tb), ob, fb);
    if (!poll_cells<4>(p, rm, oa, fa) || !poll_cells<4>(p, rm, ob, fb)) return false;
    far_push(L, pdv, ta, fa);
    far_push(L, pdv, tb, fb);
  }
  return true;
}

// ---------------------------------------------------------------- kernel

// One launch fills nb tables of one family (different budgets): ticket t
// takes column t / nb of table t % nb, so every table's columns are still
// handed out right to left.  nb = 1: the table of p0; else ps[0 .. nb).
// Workgroups per compute unit: as many as four waves per SIMD hold (four of
// four waves, three of five), so that 1024 columns are resident at once.
// Each column's row wave is a chain of dependent steps: more resident
// columns run more chains side by side (the 1031 columns of the ResNet-50
// table: 14% faster with four than with three, the batched sweep 20%).
template <int NP>
__global__ __launch_bounds__((NP + 1) * kWave)
__attribute__((amdgpu_waves_per_eu((wide_slots_per_cu(NP) * (NP + 1) + 3) / 4))) void k_fill_wide(WParams p0,
                                                                        const WParams* ps,
                                                                        int32_t nb) {
  __shared__ __attribute__((aligned(16))) uint32_t s_part[NP][kJB / 2 * 4][kWave];
  __shared__ __attribute__((aligned(16))) RowLds s_rows;
  __shared__ int32_t s_col, s_abort;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x & (kWave - 1);
  // the row wave is a chain of short dependent steps while the panel waves
  // stream packed VALU work: the row wave issues first
  if (wave == 0) __builtin_amdgcn_s_setprio(3);
  const u16x2 kInf2 = (u16x2)((unsigned short)kInfM);
  const uint32_t kInfPair = 0xFFFFFFFFu;
  while (true) {
    if (threadIdx.x == 0) {
      s_col = atomicAdd(p0.ticket, 1);
      s_abort = 0;
    }
    if (wave == 0)
#pragma unroll
      for (int q = 0; q < kJB / 2; q++)
#pragma unroll
        for (int k = 0; k < 4; k++) s_rows.nxt[q][lane + 64 * k] = kInfPair;
    __syncthreads();
    const int32_t tk = __builtin_amdgcn_readfirstlane(s_col);
    if (tk >= p0.K * nb) return;
    const int32_t c = tk / nb;
    const WParams p = batch_params(p0, ps, nb, tk);
    const int32_t cC = c * kWC;
    cint32* const meta = (cint32*)p.meta;
    cint64* const rptr = (cint64*)p.rptr;
    cint32* const live = (cint32*)p.live;
    Acc nx;                                         // a panel wave's partial minima
    acc_fill(nx, kInf2);
    // cycle b: the row wave finishes block b (b >= 0) while the panel waves
    // stream the panel of block b + 1; then the partials meet
    for (int32_t b = -1; b < p.nblk; b++) {
      const int32_t pb = b + 1;
      bool ok = true;
      jitter_delay(p.jitter, c, b, wave);
      if (wave == 0) {
        if (b >= 0) {
          const int32_t nrows = meta[b * kWMeta + 2];
          int32_t pdv = load_push(p, b, 0);
          for (int s = 0; s < nrows && ok; s++) {
            const int32_t cur = pdv;
            if (s + 1 < nrows) pdv = load_push(p, b, s + 1);    // the next row's list, early
            ok = row_step(p, c, s, cur, s_rows);
          }
        }
      } else if (pb < p.nblk) {
        cint32* mt = meta + pb * kWMeta;
        if (cC <= mt[3]) {                               // a target of block pb has cells here
          const int32_t n = live[(int64_t)pb * p.K + c];
          if (n > 0) {
            ok = gate(p, c, mt[1], mt[4]);
            if (ok) panel_records<NP>(p, wave - 1, rptr[pb], n, 2 * cC, nx);
          }
        }
      }
      if (!ok && lane == 0) s_abort = 1;
      if (wave > 0) {
#pragma unroll
        for (int q = 0; q < kJB / 2; q++)
#pragma unroll
          for (int k = 0; k < 4; k++)
            s_part[wave - 1][q * 4 + k][lane] = __builtin_bit_cast(uint32_t, nx.v[q][k]);
        acc_fill(nx, kInf2);
      } else {
        wait_vm<0>();                                  // the block's stores have completed
      }
      __syncthreads();
      if (wave == 0) {
        // the next block starts from the panel partials and the pushes
#pragma unroll
        for (int q = 0; q < kJB / 2; q++)
#pragma unroll
          for (int k = 0; k < 4; k++) {
            u16x2 m = __builtin_bit_cast(u16x2, s_rows.nxt[q][lane + 64 * k]);
#pragma unroll
            for (int w = 0; w < NP; w++)
              m = __builtin_elementwise_min(m, __builtin_bit_cast(u16x2, s_part[w][q * 4 + k][lane]));
            s_rows.acc[q][lane + 64 * k] = __builtin_bit_cast(uint32_t, m);
            s_rows.nxt[q][lane + 64 * k] = kInfPair;
          }
        jitter_delay(p.jitter, c, b, NP + 1);
        if (b >= 0 && lane == 0)
          __hip_atomic_store(&p.progress[c], 1 + (b + 1) * kJB < p.F ? 1 + (b + 1) * kJB : p.F,
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      const int32_t abort = s_abort;
      __syncthreads();
      if (abort) {
        if (threadIdx.x == 0) p.st->error = 3;
        return;
      }
    }
  }
}

__global__ void k_wide_init(int32_t* progress, int32_t K, int32_t* ticket) {
  for (int32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < K; k += gridDim.x * blockDim.x)
    progress[k] = 1;                        // the empty set's row is written by the init kernel
  if (blockIdx.x == 0 && threadIdx.x == 0) *ticket = 0;
}

// ------------------------------------------------------------ preparation
// Distinct shifts among the slots of e[kJB] (e >= 0) whose bit is set in
// mask; returns their number and writes them in ascending order.
__device__ int distinct_shifts(const int32_t* e, uint32_t mask, int32_t* out) {
  int n = 0;
  for (int s = 0; s < kJB; s++) {
    if (!((mask >> s) & 1) || e[s] < 0) continue;
    bool seen = false;
    for (int x = 0; x < n; x++) seen |= out[x] == e[s];
    if (!seen) out[n++] = e[s];
  }
  for (int x = 1; x < n; x++)
    for (int y = x; y > 0 && out[y] < out[y - 1]; y--) {
      const int32_t t = out[y];
      out[y] = out[y - 1];
      out[y - 1] = t;
    }
  return n;
}

// First source after the sources of panel(b): the rows before the previous
// block (at least the empty set).
__device__ __forceinline__ int64_t panel_end(int64_t b) {
  return b >= 1 ? 1 + (b - 1) * kJB : 1;
}

// Family time: an upper bound of the records of each block (every existing
// pair, any budget).
__global__ __launch_bounds__(256) void k_wide_count(const int64_t* rec_ptr, BlockRecords R,
                                                    int64_t* count) {
  const int64_t b = blockIdx.x;
  __shared__ unsigned long long s_n;
  if (threadIdx.x == 0) s_n = 0;
  __syncthreads();
  uint64_t n = 0;
  const int64_t end = panel_end(b);
  for (int64_t r = rec_ptr[b] + threadIdx.x; r < rec_ptr[b + 1]; r += blockDim.x) {
    if (R.src[r] >= end) continue;
    int32_t sh[kJB];
    n += distinct_shifts(R.e + r * kJB, 0xFFu, sh);
  }
  atomicAdd(&s_n, (unsigned long long)n);
  __syncthreads();
  if (threadIdx.x == 0) count[b] = (int64_t)s_n;
}

// Per solve: the live records of block b (slot with a pair and B - c >= 0),
// one per distinct shift, unsorted, from wptr[b] on: {cm, base, lim} into key
// and bl_tmp, budgets and additions into td_tmp.  meta[b] = {records, reach,
// rows, largest P of the rows, sources' end, ...}.
__global__ __launch_bounds__(256) void k_wide_prepare(int32_t F, int32_t Beff, const int32_t* w,
                                                      const int64_t* row_off,
                                                      const int64_t* rec_ptr, BlockRecords R,
                                                      const int64_t* wptr, int64_t* key,
                                                      int32_t* bl_tmp, int32_t* td_tmp,
                                                      int32_t* meta) {
  const int64_t b = blockIdx.x;
  const int64_t end = panel_end(b);
  __shared__ int32_t s_n, s_emax;
  if (threadIdx.x == 0) {
    s_n = 0;
    s_emax = 0;
  }
  __syncthreads();
  const int64_t base = wptr[b];
  for (int64_t r = rec_ptr[b] + threadIdx.x; r < rec_ptr[b + 1]; r += blockDim.x) {
    const int32_t i = R.src[r];
    if (i >= end) continue;
    uint32_t livemask = 0;
    for (int s = 0; s < kJB; s++)
      if (R.e[r * kJB + s] >= 0 && Beff - R.c[r * kJB + s] >= 0) livemask |= 1u << s;
    int32_t sh[kJB];
    const int nsh = distinct_shifts(R.e + r * kJB, livemask, sh);
    const int32_t Pi = w[i] - 1;
    const int64_t endi = row_off[i] + Pi;
    for (int x = 0; x < nsh; x++) {
      const int32_t e = sh[x];
      const int32_t o = atomicAdd(&s_n, 1);
      const int64_t d = base + o;
      uint32_t tau2[kJB / 2] = {0, 0, 0, 0}, dm2[kJB / 2] = {0, 0, 0, 0};
      for (int s = 0; s < kJB; s++) {
        const bool ok = ((livemask >> s) & 1) && R.e[r * kJB + s] == e;
        const uint32_t tv = ok ? (uint32_t)(Beff - R.c[r * kJB + s]) : 0u;
        const uint32_t dv = ok ? (R.kadd[r * kJB + s] >> 16) : 0xFFFFu;
        tau2[s / 2] |= tv << (16 * (s & 1));
        dm2[s / 2] |= dv << (16 * (s & 1));
      }
      const int64_t cm = ((int64_t)Pi + e) / kWC;        // last column the window reaches
      key[d] = (cm << 20) | (int64_t)o;
      bl_tmp[2 * d] = (int32_t)(2 * (endi + e - kWC + 1));
      bl_tmp[2 * d + 1] = (int32_t)(2 * (endi + 1));
      for (int q = 0; q < kJB / 2; q++) {
        td_tmp[d * kWTd + q] = (int32_t)tau2[q];
        td_tmp[d * kWTd + 4 + q] = (int32_t)dm2[q];
      }
      atomicMax(&s_emax, e);
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int64_t j0 = 1 + b * kJB, j1 = min<int64_t>(j0 + kJB, F);
    int32_t mp = -1;
    for (int64_t j = j0; j < j1; j++) mp = max(mp, w[j] - 1);
    int32_t* mt = meta + b * kWMeta;
    mt[0] = s_n;
    mt[1] = (s_emax + kWC - 1) / kWC + 1;           // columns to the right the windows reach
    mt[2] = (int32_t)(j1 - j0);
    mt[3] = mp;
    mt[4] = (int32_t)end;                           // rows the panel reads
    for (int x = 5; x < kWMeta; x++) mt[x] = 0;
  }
}

// Per solve: sort block b's records by the last column they reach,
// descending (bitonic sort in LDS of at most kWMaxRec keys), write them in
// that order to bl / td, and live[b * K + x] = the records reaching column x.
__global__ __launch_bounds__(256) void k_wide_sort(int32_t K, const int64_t* wptr,
                                                   const int64_t* key, const int32_t* bl_tmp,
                                                   const int32_t* td_tmp, const int32_t* meta,
                                                   int32_t* bl, int32_t* td, int32_t* live) {
  __shared__ int64_t s_key[kWMaxRec];
  const int64_t b = blockIdx.x;
  const int64_t base = wptr[b];
  const int32_t n = meta[b * kWMeta];
  int32_t N = 1;
  while (N < n) N <<= 1;
  for (int32_t x = threadIdx.x; x < N; x += blockDim.x)
    s_key[x] = x < n ? ((((int64_t)1 << 23) - 1 - (key[base + x] >> 20)) << 20) |
                           (key[base + x] & 0xFFFFF)
                     : INT64_MAX;                      // ascending key = descending column
  __syncthreads();
  for (int32_t kk = 2; kk <= N; kk <<= 1)
    for (int32_t j = kk >> 1; j > 0; j >>= 1) {
      for (int32_t x = threadIdx.x; x < N; x += blockDim.x) {
        const int32_t y = x ^ j;
        if (y > x) {
          const bool up = (x & kk) == 0;
          const int64_t a = s_key[x], c = s_key[y];
          if ((a > c) == up) {
            s_key[x] = c;
            s_key[y] = a;
          }
        }
      }
      __syncthreads();
    }
  for (int32_t x = threadIdx.x; x < n; x += blockDim.x) {
    const int64_t src = base + (s_key[x] & 0xFFFFF);
    const int64_t d = base + x;
    bl[2 * d] = bl_tmp[2 * src];
    bl[2 * d + 1] = bl_tmp[2 * src + 1];
    for (int q = 0; q < kWTd; q++) td[d * kWTd + q] = td_tmp[src * kWTd + q];
  }
  // live[x]: records whose last column is >= x (a prefix of the sorted list)
  for (int32_t x = threadIdx.x; x < K; x += blockDim.x) {
    int32_t lo = 0, hi = n;                              // first record with cm < x
    while (lo < hi) {
      const int32_t mid = (lo + hi) >> 1;
      const int64_t cm = ((int64_t)1 << 23) - 1 - (s_key[mid] >> 20);
      if (cm >= x)
        lo = mid + 1;
      else
        hi = mid;
    }
    live[b * (int64_t)K + x] = lo;
  }
}

// Per solve, row pushes: for row s of block b (source j = j0 + s) the
// targets are the later rows of the block (slots 0..7, only s2 > s) and the
// rows of block b + 1 (slots 8..15).  List layout: see kWp*.
__global__ __launch_bounds__(64) void k_wide_push(int64_t F, int64_t nblk, int32_t Beff,
                                                  const int32_t* w, const int64_t* row_off,
                                                  const int64_t* rec_ptr, BlockRecords R,
                                                  int32_t* push) {
  const int64_t b = blockIdx.x;
  const int s = threadIdx.x;
  if (s >= kJB) return;
  const int64_t j0 = 1 + b * kJB;
  const int64_t j = j0 + s;
  int32_t* d = push + (b * kJB + s) * kWPush;
  int32_t e[2 * kJB], tau[2 * kJB], dm[2 * kJB];
  for (int t = 0; t < 2 * kJB; t++) {
    e[t] = -1;
    tau[t] = 0;
    dm[t] = 0xFFFF;
  }
  if (j < F) {
    for (int s2 = s + 1; s2 < kJB && j0 + s2 < F; s2++) {      // later rows of the block
      const int64_t x = b * kJB * kJB + s * kJB + s2;
      const int32_t tv = Beff - R.tri_c[x];
      if (R.tri_e[x] >= 0 && tv >= 0) {
        e[s2] = R.tri_e[x];
        tau[s2] = tv;
        dm[s2] = (int32_t)(R.tri_kadd[x] >> 16);
      }
    }
    if (b + 1 < nblk) {                   // rows of the next block: its record of source j
      for (int64_t r = rec_ptr[b + 2] - 1; r >= rec_ptr[b + 1] && R.src[r] >= j0; r--) {
        if (R.src[r] != j) continue;
        for (int s2 = 0; s2 < kJB; s2++) {
          const int32_t ev = R.e[r * kJB + s2];
          const int32_t tv = Beff - R.c[r * kJB + s2];
          if (ev >= 0 && tv >= 0) {
            e[kJB + s2] = ev;
            tau[kJB + s2] = tv;
            dm[kJB + s2] = (int32_t)(R.kadd[r * kJB + s2] >> 16);
          }
        }
        break;
      }
    }
  }
  for (int x = 0; x < kWPush; x++) d[x] = 0;
  int32_t emax = -1, maxPt = -1, hnear = 0;
  uint32_t far = 0, near_pairs = 0;
  for (int t = 0; t < 2 * kJB; t++) {
    d[kWpE + t] = e[t];
    if (e[t] < 0) continue;
    const int64_t jt = t < kJB ? j0 + t : j0 + t;     // slot t of the next block is j0 + kJB + t - kJB
    maxPt = max(maxPt, w[jt] - 1);
    emax = max(emax, e[t]);
    if (e[t] <= kWH) {
      hnear = max(hnear, e[t]);
      near_pairs |= 1u << (t >> 1);
    } else {
      far |= 1u << t;
    }
  }
  for (int q = 0; q < kJB; q++) {
    d[kWpTau + q] = (int32_t)((uint32_t)tau[2 * q] | ((uint32_t)tau[2 * q + 1] << 16));
    d[kWpDm + q] = (int32_t)((uint32_t)dm[2 * q] | ((uint32_t)dm[2 * q + 1] << 16));
  }
  const int32_t Pj = j < F ? w[j] - 1 : -1;
  const int64_t endj = j < F ? row_off[j] + Pj : 0;
  d[kWpP] = Pj;
  d[kWpEnd] = (int32_t)(endj & 0xFFFFFFFF);
  d[kWpEnd + 1] = (int32_t)(endj >> 32);
  d[kWpEmax] = emax;
  d[kWpMaxPt] = maxPt;
  d[kWpHalo] = hnear > 0 ? (hnear + 63) / 64 * 64 : 0;
  d[kWpFar] = (int32_t)far;
  d[kWpNear] = (int32_t)near_pairs;
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

// Panel waves per workgroup for a launch of `cols` columns (all tables).
// Three while every column fits on the GPU at once with four workgroups per
// compute unit; beyond that one, so that eight workgroups fit per compute
// unit and twice as many row chains run side by side, each column's panel
// on one wave (config 3's 32-budget sweep: fill 7.4 ms against 9.3 with
// two panel waves and 10.6 with three; config 3's single table, 1031
// columns: 0.61 ms against 0.63; config 4, 720 columns, keeps three:
// 1.74 ms against 2.30 with one).
int wide_panel_waves(int64_t cols) {
  const char* env = std::getenv("RCDP_WIDE_NP");
  if (env && env[0] >= '1' && env[0] <= '4') return env[0] - '0';
  return cols > (int64_t)wide_slots_per_cu(3) * num_cus() ? 1 : 3;
}

}  // namespace

int64_t wide_columns(rc_family f) { return (f->max_row + kWC - 1) / kWC; }

hipError_t launch_wide_count(rc_family f, int64_t* count, hipStream_t s) {
  hipLaunchKernelGGL(k_wide_count, dim3((unsigned)f->nblk), dim3(256), 0, s, f->rec_ptr, f->rec,
                     count);
  return hipGetLastError();
}

// Per-table preparation (records, pushes, progress) and kernel parameters.
static hipError_t prepare_wide(rc_solution sol, int32_t K, int32_t* ticket, WParams* prm,
                               hipStream_t s) {
  rc_family f = sol->f;
  hipLaunchKernelGGL(k_wide_init, dim3((K + 255) / 256), dim3(256), 0, s, sol->progress, K,
                     ticket);
  hipError_t pe = launch_fill_pending(sol, s);
  if (pe == hipSuccess) pe = launch_pad_init(sol, s);
  if (pe != hipSuccess) return pe;
  const int64_t R = f->wrec_total;
  hipLaunchKernelGGL(k_wide_prepare, dim3((unsigned)f->nblk), dim3(256), 0, s, (int32_t)f->F,
                     (int32_t)sol->Beff, f->w, f->row_off, f->rec_ptr, f->rec, f->wrec_ptr,
                     sol->wkey, sol->wbl_tmp, sol->wtd_tmp, sol->wmeta);
  hipLaunchKernelGGL(k_wide_sort, dim3((unsigned)f->nblk), dim3(256), 0, s, K, f->wrec_ptr,
                     sol->wkey, sol->wbl_tmp, sol->wtd_tmp, sol->wmeta, sol->wbl, sol->wtd,
                     sol->wlive);
  hipLaunchKernelGGL(k_wide_push, dim3((unsigned)f->nblk), dim3(64), 0, s, f->F, f->nblk,
                     (int32_t)sol->Beff, f->w, f->row_off, f->rec_ptr, f->rec, sol->wpush);
  pe = hipGetLastError();
  if (pe != hipSuccess) return pe;
  prm->F = (int32_t)f->F;
  prm->nblk = (int32_t)f->nblk;
  prm->K = K;
  prm->meta = sol->wmeta;
  prm->rptr = f->wrec_ptr;
  prm->live = sol->wlive;
  prm->bl = sol->wbl;
  prm->td = sol->wtd;
  prm->rec_cap = (int32_t)R;
  prm->push = sol->wpush;
  prm->m = sol->m;
  prm->m_bytes = 2 * f->cells_alloc;
  prm->null_off = (int32_t)(2 * f->cells);         // the trailing guard: kGuard infinite cells
  prm->progress = sol->progress;
  prm->ticket = ticket;
  prm->st = sol->status;
  prm->timeout_ticks = wait_ticks();
  prm->jitter = jitter_seed();
  return hipSuccess;
}

static hipError_t launch_wide_kernel(const WParams& prm, const WParams* dev, int32_t nb,
                                     hipEvent_t e0, hipEvent_t e1, hipStream_t s) {
  const int64_t cols = (int64_t)prm.K * nb;
  const int np = wide_panel_waves(cols);
  const int32_t grid = (int32_t)std::min<int64_t>(cols, (int64_t)num_cus() * wide_slots_per_cu(np));
  if (std::getenv("RCDP_DEBUG"))
    std::fprintf(stderr, "rcdp: split-panel fill %d table(s) x K=%d columns of %d cells, "
                 "grid=%d, %d panel waves\n", nb, prm.K, kWC, grid, np);
  if (e0 && hipEventRecord(e0, s) != hipSuccess) return hipErrorUnknown;
  if (np == 4)
    hipLaunchKernelGGL(k_fill_wide<4>, dim3(grid), dim3(5 * kWave), 0, s, prm, dev, nb);
  else if (np == 2)
    hipLaunchKernelGGL(k_fill_wide<2>, dim3(grid), dim3(3 * kWave), 0, s, prm, dev, nb);
  else if (np == 1)
    hipLaunchKernelGGL(k_fill_wide<1>, dim3(grid), dim3(2 * kWave), 0, s, prm, dev, nb);
  else
    hipLaunchKernelGGL(k_fill_wide<3>, dim3(grid), dim3(4 * kWave), 0, s, prm, dev, nb);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (e1 && hipEventRecord(e1, s) != hipSuccess) return hipErrorUnknown;
  return hipSuccess;
}

hipError_t launch_fill_wide(rc_solution sol, hipStream_t s) {
  rc_family f = sol->f;
  if (f->F < 2) return hipSuccess;
  const int32_t K = (int32_t)wide_columns(f);
  WParams prm;
  const hipError_t pe = prepare_wide(sol, K, sol->ticket, &prm, s);
  if (pe != hipSuccess) return pe;
  return launch_wide_kernel(prm, nullptr, 1, sol->evk0, sol->evk1, s);
}

hipError_t launch_fill_wide_batch(rc_solution* sols, int32_t nb, WParams* host_prm,
                                  WParams* dev_prm, hipStream_t s) {
  rc_family f = sols[0]->f;
  if (f->F < 2) return hipSuccess;
  const int32_t K = (int32_t)wide_columns(f);
  for (int32_t b = 0; b < nb; b++) {
    // every table resets the shared ticket; they all run before the kernel
    const hipError_t pe = prepare_wide(sols[b], K, sols[0]->ticket, &host_prm[b], s);
    if (pe != hipSuccess) return pe;
  }
  const hipError_t ce = hipMemcpyAsync(dev_prm, host_prm, sizeof(WParams) * (size_t)nb,
                                       hipMemcpyHostToDevice, s);
  if (ce != hipSuccess) return ce;
  return launch_wide_kernel(host_prm[0], dev_prm, nb, sols[0]->evk0, sols[0]->evk1, s);
}

}  // namespace rcdp
