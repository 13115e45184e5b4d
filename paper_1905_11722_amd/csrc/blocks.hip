// Target-block records for the blocked wavefront fill (blocked.hip).
//
// Targets 1..F-1 (family order) are cut into blocks of at most kJB
// consecutive targets, block b = [bstart[b], bstart[b + 1]): kJB targets
// each for the row-push wavefront (blocked.hip), blocks whose in-block
// dependencies fit the recomputed halo for the ghost-zone wavefront
// (ghost.hip).  For block b = [j0, j1) the pairs (L_i, L_j) with j in the
// block split into
//  - panel pairs, i < j0: grouped into one record per source i (ascending
//    i), holding kJB slots (one per target of the block; e = -1 when the
//    pair does not exist);
//  - triangle pairs, j0 <= i < j: a kJB x kJB matrix per block.
// A slot stores the pair's right-aligned shift e, its packed key addend
// (dm << 16 | i) and its budget term c.  With P_L = w_L - 1 = T(L \ bd(L)),
// the step t' = t + dt of Algorithm 1 maps the cell at distance u = t - P_i
// from the end of row i to distance u' = u - e from the end of row j, where
// e = P_j - P_i - dt = T(bd(L_i) \ bd(L_j)) >= 0: only boundary nodes of
// L_i that L_j closes move a cell relative to the row ends.  Consecutive
// targets mostly close the same nodes, so e barely changes across a block,
// and one window of source row i serves every target of the block.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "rc_internal.h"

namespace rcdp {

namespace {

// Number of panel sources (distinct i < j0 over the block's pred lists).
__global__ __launch_bounds__(256) void k_blk_count(const int32_t* bstart, const int64_t* pred_ptr,
                                                   const int32_t* pidx, int64_t* count) {
  __shared__ uint32_t bitmap[(kMaxSets + 32) / 32];
  __shared__ int32_t total;
  const int64_t b = blockIdx.x;
  const int64_t j0 = bstart[b], j1 = bstart[b + 1];
  const int words = (int)((j0 + 31) / 32);
  for (int x = threadIdx.x; x < words; x += blockDim.x) bitmap[x] = 0;
  if (threadIdx.x == 0) total = 0;
  __syncthreads();
  for (int64_t j = j0; j < j1; j++)
    for (int64_t q = pred_ptr[j] + threadIdx.x; q < pred_ptr[j + 1]; q += blockDim.x) {
      const int32_t i = pidx[q];
      if (i < j0) atomicOr(&bitmap[i >> 5], 1u << (i & 31));
    }
  __syncthreads();
  int c = 0;
  for (int x = threadIdx.x; x < words; x += blockDim.x) c += __popc(bitmap[x]);
  atomicAdd(&total, c);
  __syncthreads();
  if (threadIdx.x == 0) count[b] = total;
}

__global__ __launch_bounds__(256) void k_blk_fill(const int32_t* bstart, const int32_t* w,
                                                  const int64_t* pred_ptr, const int32_t* pidx,
                                                  const int32_t* pdt, const int32_t* pdm,
                                                  const int32_t* pc, const int64_t* rec_ptr,
                                                  BlockRecords R) {
  __shared__ uint32_t bitmap[(kMaxSets + 32) / 32];
  __shared__ int32_t prefix[(kMaxSets + 32) / 32];
  const int64_t b = blockIdx.x;
  const int64_t j0 = bstart[b], j1 = bstart[b + 1];
  const int words = (int)((j0 + 31) / 32);
  const int64_t base = rec_ptr[b], nrec = rec_ptr[b + 1] - base;
  for (int x = threadIdx.x; x < words; x += blockDim.x) bitmap[x] = 0;
  for (int64_t x = threadIdx.x; x < nrec * kJB; x += blockDim.x) R.e[base * kJB + x] = -1;
  for (int x = threadIdx.x; x < kJB * kJB; x += blockDim.x) R.tri_e[b * kJB * kJB + x] = -1;
  __syncthreads();
  for (int64_t j = j0; j < j1; j++)
    for (int64_t q = pred_ptr[j] + threadIdx.x; q < pred_ptr[j + 1]; q += blockDim.x) {
      const int32_t i = pidx[q];
      if (i < j0) atomicOr(&bitmap[i >> 5], 1u << (i & 31));
    }
  __syncthreads();
  // exclusive prefix of the popcounts, 256 words per pass
  __shared__ int32_t s_wsum[4];
  int32_t carry = 0;
  for (int w0 = 0; w0 < words; w0 += 256) {
    const int x = w0 + (int)threadIdx.x;
    const int32_t v = x < words ? __popc(bitmap[x]) : 0;
    int32_t incl = v;
    for (int off = 1; off < 64; off <<= 1) {
      const int32_t y = __shfl_up(incl, off, 64);
      if ((threadIdx.x & 63) >= off) incl += y;
    }
    if ((threadIdx.x & 63) == 63) s_wsum[threadIdx.x / 64] = incl;
    __syncthreads();
    int32_t before = carry;
    for (int q = 0; q < (int)threadIdx.x / 64; q++) before += s_wsum[q];
    if (x < words) prefix[x] = before + incl - v;
    carry += s_wsum[0] + s_wsum[1] + s_wsum[2] + s_wsum[3];
    __syncthreads();
  }
  for (int64_t j = j0; j < j1; j++) {
    const int slot = (int)(j - j0);
    for (int64_t q = pred_ptr[j] + threadIdx.x; q < pred_ptr[j + 1]; q += blockDim.x) {
      const int32_t i = pidx[q];
      const int32_t e = (w[j] - w[i]) - pdt[q];       // T(bd(L_i) \ bd(L_j))
      const uint32_t kadd = ((uint32_t)pdm[q] << 16) | (uint32_t)i;
      if (i < j0) {
        const int32_t rank =
            prefix[i >> 5] + __popc(bitmap[i >> 5] & ((1u << (i & 31)) - 1u));
        const int64_t r = base + rank;
        R.src[r] = i;
        R.e[r * kJB + slot] = e;
        R.kadd[r * kJB + slot] = kadd;
        R.c[r * kJB + slot] = pc[q];
      } else {
        const int64_t t = b * kJB * kJB + (int64_t)(i - j0) * kJB + slot;
        R.tri_e[t] = e;
        R.tri_kadd[t] = kadd;
        R.tri_c[t] = pc[q];
      }
    }
  }
}

}  // namespace

hipError_t launch_blk_count(rc_family f, int64_t nblk, int64_t* count, hipStream_t s) {
  hipLaunchKernelGGL(k_blk_count, dim3((unsigned)nblk), dim3(256), 0, s, f->bstart, f->pred_ptr,
                     f->pidx, count);
  return hipGetLastError();
}

hipError_t launch_blk_fill(rc_family f, int64_t nblk, hipStream_t s) {
  hipLaunchKernelGGL(k_blk_fill, dim3((unsigned)nblk), dim3(256), 0, s, f->bstart, f->w, f->pred_ptr,
                     f->pidx, f->pdt, f->pdm, f->pc, f->rec_ptr, f->rec);
  return hipGetLastError();
}

}  // namespace rcdp

namespace rcdp {

namespace {

// Shift clusters of a record: its slots sorted by shift, cut wherever the
// shift exceeds the first shift of the current cluster by more than kSpan.
// Each cluster becomes one compact record, so a staged window of
// C + kSpan cells serves every slot of it.  Returns the count and fills
// cl[s] (cluster number of slot s, -1 without a pair).
__device__ int record_clusters(const int32_t* e, int32_t* cl) {
  int32_t order[kJB];
  int n = 0;
  for (int s = 0; s < kJB; s++) {
    cl[s] = -1;
    if (e[s] >= 0) order[n++] = s;
  }
  for (int x = 1; x < n; x++)            // insertion sort by shift
    for (int y = x; y > 0 && e[order[y]] < e[order[y - 1]]; y--) {
      const int32_t t = order[y];
      order[y] = order[y - 1];
      order[y - 1] = t;
    }
  int ncl = 0;
  int32_t first = 0;
  for (int x = 0; x < n; x++) {
    const int32_t ev = e[order[x]];
    if (x == 0 || ev - first > kSpan) {
      first = ev;
      ncl++;
    }
    cl[order[x]] = ncl - 1;
  }
  return ncl;
}

// Compact records per block (B-independent upper bound for every solve).
__global__ __launch_bounds__(256) void k_blk_clusters(const int64_t* rec_ptr, BlockRecords R,
                                                      int64_t* count) {
  const int64_t b = blockIdx.x;
  __shared__ int64_t s_n;
  if (threadIdx.x == 0) s_n = 0;
  __syncthreads();
  int64_t n = 0;
  for (int64_t r = rec_ptr[b] + threadIdx.x; r < rec_ptr[b + 1]; r += blockDim.x) {
    int32_t cl[kJB];
    n += record_clusters(R.e + r * kJB, cl);
  }
  atomicAdd((unsigned long long*)&s_n, (unsigned long long)n);
  __syncthreads();
  if (threadIdx.x == 0) count[b] = s_n;
}

// Per solve, panel records: keep the slots whose budget test can pass
// (pair exists and B - c >= 0) of the records whose source lies before the
// previous block (row-push fill: sources i < bstart[b - 1], the previous
// block's rows reach the block through row pushes instead) or before the
// block itself (ghost-zone fill: every source i < j0), and emit one compact record
// per shift cluster that has such a slot, compacted from clu_ptr[b] on.  A
// compact record is kRecInts int32: [0] source i, [1] smallest shift emin,
// [2] staged span emax - emin (<= kSpan), [3] P_i = w_i - 1, [4..5] index of
// the cell u = 0 of row i (int64), [6] emax, [7] a = emin mod 8 (the
// window starts on a 16-byte boundary, a cells before the cell of shift
// emin), [8 + s] a + shift - emin of slot s (its cell in the window),
// [16 + p] budgets B - c of slots 2p, 2p+1 as two uint16, [20 + p] the
// additions dm of slots 2p, 2p+1 as two uint16, [24 .. 29] the window DMA
// terms that do not depend on the column: [24 .. 25] base = the cell u = 0
// of row i + emin - a (int64), [26] the cells of row i's 64-aligned slot,
// [27] emin - a, [28] emin, [29] emax + P_i.  A slot without a live pair
// gets budget 0 and addition 0xFFFF, so its candidate always saturates to
// infinity.  meta[b * kMetaInts] = {records, largest live shift, rows of
// the block, largest P of its rows, (set by k_rec_sort), largest live
// shift of the new group, 0, 0}; with ghost set, [1] covers the records of
// sources before the previous block (the old group) and [5] those of the
// previous block's rows (the new group).
__global__ __launch_bounds__(256) void k_rec_prepare(const int32_t* bstart, int32_t ghost,
                                                     int32_t Beff, const int32_t* w,
                                                     const int64_t* row_off,
                                                     const int64_t* rec_ptr,
                                                     const int64_t* clu_ptr, BlockRecords R,
                                                     int32_t* crec, int32_t* meta) {
  const int64_t b = blockIdx.x;
  const int64_t base = rec_ptr[b], n = rec_ptr[b + 1] - base;
  const int64_t obase = clu_ptr[b];
  const int64_t j0 = bstart[b];
  const int64_t prev = b > 0 ? bstart[b - 1] : 0;    // first row of the previous block
  const int64_t old_end = ghost ? j0 : (prev > 1 ? prev : 1);
  const int lane = threadIdx.x & 63, wave = threadIdx.x / 64;
  __shared__ int32_t s_wcnt[4];
  __shared__ int32_t s_run, s_emax, s_emax_new;
  if (threadIdx.x == 0) {
    s_run = 0;
    s_emax = 0;
    s_emax_new = 0;
  }
  __syncthreads();
  for (int64_t r0 = 0; r0 < n; r0 += 256) {
    const int64_t r = r0 + threadIdx.x;
    int32_t e[kJB], cl[kJB];
    int ncl = 0;
    uint32_t live_cl = 0;                  // clusters with a live slot
    if (r < n && R.src[base + r] < old_end) {
      for (int s = 0; s < kJB; s++) e[s] = R.e[(base + r) * kJB + s];
      ncl = record_clusters(e, cl);
      for (int s = 0; s < kJB; s++)
        if (cl[s] >= 0 && Beff - R.c[(base + r) * kJB + s] >= 0) live_cl |= 1u << cl[s];
    }
    const int mine = __popc(live_cl);
    int incl = mine;                       // inclusive prefix over the workgroup
    for (int off = 1; off < 64; off <<= 1) {
      const int y = __shfl_up(incl, off, 64);
      if (lane >= off) incl += y;
    }
    if (lane == 63) s_wcnt[wave] = incl;
    __syncthreads();
    int32_t o = s_run + incl - mine;
    for (int q = 0; q < wave; q++) o += s_wcnt[q];
    for (int k = 0; k < ncl; k++) {
      if (!(live_cl & (1u << k))) continue;
      int32_t* d = crec + (obase + o) * kRecInts;
      const int32_t i = R.src[base + r];
      const int32_t Pi = w[i] - 1;
      const int64_t endi = row_off[i] + Pi;
      int32_t emin = INT32_MAX, emax = -1;
      for (int s = 0; s < kJB; s++)
        if (cl[s] == k) {
          emin = min(emin, e[s]);
          emax = max(emax, e[s]);
        }
      uint32_t tau2[kJB / 2] = {0, 0, 0, 0}, dm2[kJB / 2] = {0, 0, 0, 0};
      for (int s = 0; s < kJB; s++) {
        const int32_t tau = Beff - R.c[(base + r) * kJB + s];
        const bool ok = cl[s] == k && tau >= 0;
        d[8 + s] = (emin & 7) + (ok ? e[s] - emin : 0);
        const uint32_t tv = ok ? (uint32_t)tau : 0u;
        const uint32_t dv = ok ? (R.kadd[(base + r) * kJB + s] >> 16) : 0xFFFFu;
        tau2[s / 2] |= tv << (16 * (s & 1));
        dm2[s / 2] |= dv << (16 * (s & 1));
      }
      d[0] = i;
      d[1] = emin;
      d[2] = emax - emin;
      d[3] = Pi;
      d[4] = (int32_t)(endi & 0xFFFFFFFF);
      d[5] = (int32_t)(endi >> 32);
      d[6] = emax;
      d[7] = emin & 7;
      for (int x = 0; x < kJB / 2; x++) {
        d[16 + x] = (int32_t)tau2[x];
        d[20 + x] = (int32_t)dm2[x];
      }
      const int64_t base_cell = endi + emin - (emin & 7);
      d[kRecDma + 0] = (int32_t)(base_cell & 0xFFFFFFFF);
      d[kRecDma + 1] = (int32_t)(base_cell >> 32);
      d[kRecDma + 2] = (int32_t)((Pi + kRowAlign) / kRowAlign * kRowAlign);
      d[kRecDma + 3] = emin - (emin & 7);
      d[kRecDma + 4] = emin;
      d[kRecDma + 5] = emax + Pi;
      for (int x = kRecDma + 6; x < kRecInts; x++) d[x] = 0;
      atomicMax(ghost && i >= prev ? &s_emax_new : &s_emax, emax);
      o++;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int32_t t = 0;
      for (int q = 0; q < 4; q++) t += s_wcnt[q];
      s_run += t;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const int64_t j1 = bstart[b + 1];
    int32_t mp = -1;
    for (int64_t j = j0; j < j1; j++) mp = max(mp, w[j] - 1);
    int32_t* mt = meta + b * kMetaInts;
    mt[0] = s_run;                      // live panel records
    mt[1] = s_emax;                     // largest live panel shift (old group)
    mt[2] = (int32_t)(j1 - j0);         // rows of the block
    mt[3] = mp;                         // largest P of the block's rows
    mt[4] = 0;
    mt[5] = s_emax_new;                 // largest live shift of the new group
    for (int x = 6; x < kMetaInts; x++) mt[x] = 0;
  }
}

// Per solve, row pushes: for row s of block b (source j = j0 + s) the
// targets are the later rows of the block (slots 0..7, only s2 > s) and the
// rows of block b + 1 (slots 8..15).  A live target (pair exists, B - c >= 0)
// with shift e <= kHalo reads the source row buffer at offset e (own column
// plus halo); a larger shift gets a staged window of its own.  List layout
// (kPushInts int32): [0] halo cells (largest near shift rounded up to 8),
// [1] far windows, [2] largest P over live targets (-1 none), [3] largest
// live shift, [4] P_j, [5..6] index of the cell u = 0 of row j, [8 + k] the
// shift of far window k, [24 + p] LDS cell offsets of targets 2p, 2p+1 as
// two uint16 (near: e, relative to the row buffer; far: 2 RB + k FB + e % 8
// with RB = C + kHalo + 8, FB = C + 8), [32 + p] budgets and [40 + p]
// additions of targets 2p, 2p+1 as two uint16 (dead: 0 and 0xFFFF).
__global__ __launch_bounds__(64) void k_push_prepare(int64_t F, int64_t nblk, int32_t Beff,
                                                     int32_t C, const int32_t* w,
                                                     const int64_t* row_off,
                                                     const int64_t* rec_ptr, BlockRecords R,
                                                     int32_t* push) {
  const int64_t b = blockIdx.x;
  const int s = threadIdx.x;
  if (s >= kJB) return;
  const int64_t j0 = 1 + b * kJB;
  const int64_t j = j0 + s;
  int32_t* d = push + (b * kJB + s) * kPushInts;
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
  const int32_t RB = C + kHalo + 8, FB = C + 8;
  int32_t hs = 0, nfar = 0, maxPt = -1, emax = -1;
  int32_t off[2 * kJB];
  for (int x = 0; x < 2 * kPushInts / 2; x++) d[x] = 0;
  for (int t = 0; t < 2 * kJB; t++) {
    off[t] = 0;
    if (e[t] < 0) continue;
    const int64_t jt = t < kJB ? j0 + t : j0 + kJB + (t - kJB);
    maxPt = max(maxPt, w[jt] - 1);
    emax = max(emax, e[t]);
    if (e[t] <= kHalo) {
      off[t] = e[t];
      hs = max(hs, (e[t] + 7) / 8 * 8);
    } else {
      d[8 + nfar] = e[t];
      off[t] = 2 * RB + nfar * FB + (e[t] & 7);
      nfar++;
    }
  }
  d[0] = hs;
  d[1] = nfar;
  d[2] = maxPt;
  d[3] = emax;
  const int32_t Pj = j < F ? w[j] - 1 : -1;
  const int64_t endj = j < F ? row_off[j] + Pj : 0;
  d[4] = Pj;
  d[5] = (int32_t)(endj & 0xFFFFFFFF);
  d[6] = (int32_t)(endj >> 32);
  for (int p = 0; p < kJB; p++) {
    d[24 + p] = (int32_t)((uint32_t)off[2 * p] | ((uint32_t)off[2 * p + 1] << 16));
    d[32 + p] = (int32_t)((uint32_t)tau[2 * p] | ((uint32_t)tau[2 * p + 1] << 16));
    d[40 + p] = (int32_t)((uint32_t)dm[2 * p] | ((uint32_t)dm[2 * p + 1] << 16));
  }
}

// Per solve, order of the panel records of each block: two kinds, first
// kind 0, then kind 1; within each kind by descending
// cm = min(floor((P_i + emax + H) / C), cap - 1), the last column whose
// cells the record's window reaches (a column also computes the H cells
// to its right).  Kinds: ghost == 0, records whose slots share one shift
// ("uniform", span 0) and the rest; ghost != 0, sources before the previous
// block (old group) and the previous block's rows (new group).  For every
// column x < cap the live table holds, per kind, the number of records with
// cm >= x: a prefix of the kind's records that contains every record whose
// window reaches column x (for x = cap - 1 also columns beyond).  meta[4] =
// the number of kind-0 records.
__global__ __launch_bounds__(256) void k_rec_sort(int32_t C, int32_t H, int32_t cap,
                                                  const int32_t* bstart, int32_t ghost,
                                                  const int64_t* clu_ptr, const int32_t* src,
                                                  int32_t* dst, int32_t* meta, int32_t* live) {
  constexpr int kPer = 2 * kLiveCap / 256;       // bins per thread in the scan
  __shared__ int32_t bin[2 * kLiveCap];
  __shared__ int32_t s_part[256];
  const int64_t b = blockIdx.x;
  const int64_t base = clu_ptr[b];
  const int32_t n = meta[b * kMetaInts + 0];
  const int32_t prev = b > 0 ? bstart[b - 1] : 0;
  const int tid = threadIdx.x;
  const int nb = 2 * cap;
  for (int x = tid; x < 2 * kLiveCap; x += 256) bin[x] = 0;
  __syncthreads();
  auto key_of = [&](const int32_t* rec) {
    const int32_t cm = min((rec[3] + rec[6] + H) / C, cap - 1);
    const bool kind1 = ghost ? rec[0] >= prev : rec[2] != 0;
    return (kind1 ? cap : 0) + (cap - 1 - cm);
  };
  for (int32_t r = tid; r < n; r += 256) atomicAdd(&bin[key_of(src + (base + r) * kRecInts)], 1);
  __syncthreads();
  // exclusive prefix over the 2 * cap bins (kPer consecutive bins per thread)
  int32_t loc[kPer];
  int32_t run = 0;
  for (int x = 0; x < kPer; x++) {
    const int k = tid * kPer + x;
    loc[x] = run;
    run += k < nb ? bin[k] : 0;
  }
  s_part[tid] = run;
  __syncthreads();
  if (tid == 0) {
    int32_t acc = 0;
    for (int q = 0; q < 256; q++) {
      const int32_t v = s_part[q];
      s_part[q] = acc;
      acc += v;
    }
  }
  __syncthreads();
  for (int x = 0; x < kPer; x++) {
    const int k = tid * kPer + x;
    if (k < nb) bin[k] = s_part[tid] + loc[x];    // exclusive prefix P[k]
  }
  __syncthreads();
  // live counts: kind s, column x -> P[s cap + cap - x] - P[s cap]
  auto P = [&](int k) { return k < nb ? bin[k] : n; };
  for (int x = tid; x < cap; x += 256) {
    live[((int64_t)b * cap + x) * 2 + 0] = P(cap - x) - P(0);
    live[((int64_t)b * cap + x) * 2 + 1] = P(2 * cap - x) - P(cap);
  }
  if (tid == 0) meta[b * kMetaInts + 4] = P(cap);
  __syncthreads();
  // scatter (bins become cursors)
  for (int32_t r = tid; r < n; r += 256) {
    const int32_t* rec = src + (base + r) * kRecInts;
    const int32_t pos = atomicAdd(&bin[key_of(rec)], 1);
    int32_t* d = dst + (base + pos) * kRecInts;
    for (int x = 0; x < kRecInts; x++) d[x] = rec[x];
  }
}

// Every table cell after row 0 starts out as "not written yet".
__global__ void k_fill_pending(uint4* p, int64_t n16) {
  const uint32_t v = kPendM | (kPendM << 16);
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < n16;
       x += (int64_t)gridDim.x * blockDim.x)
    p[x] = make_uint4(v, v, v, v);
}

// The padding of every row (the cells of its slot before the row, at least
// kGuard of them), the kGuard cells after the last row and an 8-cell
// sentinel hold infinity, so that window loads that touch them read
// infinity.  One workgroup per row.
__global__ void k_pad_init(int64_t F, const int32_t* w, const int64_t* row_off, int64_t cells,
                           uint16_t* m, uint16_t* sentinel) {
  for (int64_t s = blockIdx.x; s <= F; s += gridDim.x) {
    const int64_t start = s < F ? row_off[s] + w[s] - row_slot(w[s]) : cells;
    const int64_t end = s < F ? row_off[s] : cells + kGuard;
    for (int64_t x = start + threadIdx.x; x < end; x += blockDim.x) m[x] = (uint16_t)kInfM;
  }
  if (blockIdx.x == 0 && threadIdx.x < 8 && sentinel) sentinel[threadIdx.x] = (uint16_t)kInfM;
}

}  // namespace

hipError_t launch_rec_prepare(rc_solution sol, hipStream_t s) {
  rc_family f = sol->f;
  hipLaunchKernelGGL(k_rec_prepare, dim3((unsigned)f->nblk), dim3(256), 0, s, f->bstart,
                     (int32_t)(f->blk_kind == kBlocksGhost), (int32_t)sol->Beff, f->w, f->row_off,
                     f->rec_ptr, f->clu_ptr, f->rec, sol->crec_tmp, sol->blk_meta);
  return hipGetLastError();
}

hipError_t launch_rec_sort(rc_solution sol, int32_t C, int32_t H, hipStream_t s) {
  rc_family f = sol->f;
  hipLaunchKernelGGL(k_rec_sort, dim3((unsigned)f->nblk), dim3(256), 0, s, C, H, sol->live_cap,
                     f->bstart, (int32_t)(f->blk_kind == kBlocksGhost), f->clu_ptr, sol->crec_tmp,
                     sol->crec, sol->blk_meta, sol->live);
  return hipGetLastError();
}

hipError_t launch_push_prepare(rc_solution sol, int32_t C, hipStream_t s) {
  rc_family f = sol->f;
  hipLaunchKernelGGL(k_push_prepare, dim3((unsigned)f->nblk), dim3(64), 0, s, f->F, f->nblk,
                     (int32_t)sol->Beff, C, f->w, f->row_off, f->rec_ptr, f->rec, sol->push);
  return hipGetLastError();
}

// Cells after row 0's slot (row 0, the empty set, holds its one cell).
hipError_t launch_fill_pending(rc_solution sol, hipStream_t s) {
  rc_family f = sol->f;
  const int64_t first = row_slot(1);                 // slot 0 holds the empty set's row
  const int64_t n16 = (f->cells - first) / 8;
  if (n16 <= 0) return hipSuccess;
  const unsigned grid = (unsigned)std::min<int64_t>((n16 + 255) / 256, 4096);
  hipLaunchKernelGGL(k_fill_pending, dim3(grid), dim3(256), 0, s,
                     reinterpret_cast<uint4*>(sol->m + first), n16);
  return hipGetLastError();
}

hipError_t launch_blk_clusters(rc_family f, int64_t* count, hipStream_t s) {
  hipLaunchKernelGGL(k_blk_clusters, dim3((unsigned)f->nblk), dim3(256), 0, s, f->rec_ptr, f->rec,
                     count);
  return hipGetLastError();
}

hipError_t launch_pad_init(rc_solution sol, hipStream_t s) {
  rc_family f = sol->f;
  const unsigned grid = (unsigned)std::min<int64_t>(f->F + 1, 4096);
  hipLaunchKernelGGL(k_pad_init, dim3(grid), dim3(256), 0, s, f->F, f->w, f->row_off, f->cells,
                     sol->m, sol->sentinel);
  return hipGetLastError();
}

}  // namespace rcdp
