// Target-block records for the blocked wavefront fill (blocked.hip).
//
// Targets 1..F-1 (family order) are cut into blocks of kJB consecutive
// targets.  For block b = [j0, j1) the pairs (L_i, L_j) with j in the
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

#include "rc_internal.h"

namespace rcdp {

namespace {

// Number of panel sources (distinct i < j0 over the block's pred lists).
__global__ __launch_bounds__(256) void k_blk_count(int64_t F, const int64_t* pred_ptr,
                                                   const int32_t* pidx, int64_t* count) {
  __shared__ uint32_t bitmap[(kMaxSets + 32) / 32];
  __shared__ int32_t total;
  const int64_t b = blockIdx.x;
  const int64_t j0 = 1 + b * kJB, j1 = j0 + kJB < F ? j0 + kJB : F;
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

__global__ __launch_bounds__(256) void k_blk_fill(int64_t F, const int32_t* w,
                                                  const int64_t* pred_ptr, const int32_t* pidx,
                                                  const int32_t* pdt, const int32_t* pdm,
                                                  const int32_t* pc, const int64_t* rec_ptr,
                                                  BlockRecords R) {
  __shared__ uint32_t bitmap[(kMaxSets + 32) / 32];
  __shared__ int32_t prefix[(kMaxSets + 32) / 32];
  const int64_t b = blockIdx.x;
  const int64_t j0 = 1 + b * kJB, j1 = j0 + kJB < F ? j0 + kJB : F;
  const int words = (int)((j0 + 31) / 32);
  const int64_t base = rec_ptr[b], nrec = rec_ptr[b + 1] - base;
  for (int x = threadIdx.x; x < words; x += blockDim.x) bitmap[x] = 0;
  for (int64_t r = threadIdx.x; r < nrec; r += blockDim.x) {
    R.emin[base + r] = INT32_MAX;
    R.emax[base + r] = -1;
    for (int s = 0; s < kJB; s++) R.e[(base + r) * kJB + s] = -1;
  }
  for (int x = threadIdx.x; x < kJB * kJB; x += blockDim.x) R.tri_e[b * kJB * kJB + x] = -1;
  for (int x = threadIdx.x; x < kJB; x += blockDim.x) R.tri_emax[b * kJB + x] = -1;
  if (threadIdx.x == 0) R.blk_emax[b] = 0;
  __syncthreads();
  for (int64_t j = j0; j < j1; j++)
    for (int64_t q = pred_ptr[j] + threadIdx.x; q < pred_ptr[j + 1]; q += blockDim.x) {
      const int32_t i = pidx[q];
      if (i < j0) atomicOr(&bitmap[i >> 5], 1u << (i & 31));
    }
  __syncthreads();
  if (threadIdx.x == 0) {              // exclusive prefix of popcounts
    int32_t run = 0;
    for (int x = 0; x < words; x++) {
      prefix[x] = run;
      run += __popc(bitmap[x]);
    }
  }
  __syncthreads();
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
        atomicMin(&R.emin[r], e);
        atomicMax(&R.emax[r], e);
        atomicMax(&R.blk_emax[b], e);
      } else {
        const int64_t t = b * kJB * kJB + (int64_t)(i - j0) * kJB + slot;
        R.tri_e[t] = e;
        R.tri_kadd[t] = kadd;
        R.tri_c[t] = pc[q];
        atomicMax(&R.tri_emax[b * kJB + (i - j0)], e);
      }
    }
  }
}

}  // namespace

hipError_t launch_blk_count(rc_family f, int64_t nblk, int64_t* count, hipStream_t s) {
  hipLaunchKernelGGL(k_blk_count, dim3((unsigned)nblk), dim3(256), 0, s, f->F, f->pred_ptr,
                     f->pidx, count);
  return hipGetLastError();
}

hipError_t launch_blk_fill(rc_family f, int64_t nblk, hipStream_t s) {
  hipLaunchKernelGGL(k_blk_fill, dim3((unsigned)nblk), dim3(256), 0, s, f->F, f->w, f->pred_ptr,
                     f->pidx, f->pdt, f->pdm, f->pc, f->rec_ptr, f->rec);
  return hipGetLastError();
}

}  // namespace rcdp
