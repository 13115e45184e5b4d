// Microbenchmarks of the MI355X peaks the DP fill is rated against, measured
// in the same run as the fill: the 32-bit integer VALU rate, the packed
// 16-bit integer VALU rate (two operations per lane and instruction) and the
// HBM stream bandwidth of a device-to-device copy.
//
// The VALU kernels run eight independent chains per lane of alternating add
// and min instructions, written as inline assembly so that the compiler can
// neither fold nor fuse them; every lane performs 2 * kChains operations of
// its chains per unrolled round (packed: twice as many).  The copy moves a
// buffer of 16-byte vectors, grid-strided, read once and written once.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kChains = 8;
constexpr int kUnroll = 16;

__global__ __launch_bounds__(256) void k_valu_i32(uint32_t* out, int iters, uint32_t seed) {
  const uint32_t tid = blockIdx.x * blockDim.x + threadIdx.x;
  uint32_t a[kChains];
#pragma unroll
  for (int c = 0; c < kChains; c++) a[c] = seed + tid * (c + 1);
  const uint32_t b = seed ^ 0x9E3779B9u;
  const uint32_t lim = 0xFFFFFF00u ^ seed;
  for (int i = 0; i < iters; i++) {
#pragma unroll
    for (int r = 0; r < kUnroll; r++) {
#pragma unroll
      for (int c = 0; c < kChains; c++) asm volatile("v_add_u32 %0, %0, %1" : "+v"(a[c]) : "v"(b));
#pragma unroll
      for (int c = 0; c < kChains; c++) asm volatile("v_min_u32 %0, %0, %1" : "+v"(a[c]) : "v"(lim));
    }
  }
  uint32_t x = 0;
#pragma unroll
  for (int c = 0; c < kChains; c++) x ^= a[c];
  out[tid] = x;
}

__global__ __launch_bounds__(256) void k_valu_pk_u16(uint32_t* out, int iters, uint32_t seed) {
  const uint32_t tid = blockIdx.x * blockDim.x + threadIdx.x;
  uint32_t a[kChains];
#pragma unroll
  for (int c = 0; c < kChains; c++) a[c] = seed + tid * (c + 1);
  const uint32_t b = (seed ^ 0x9E3779B9u) & 0x00FF00FFu;
  const uint32_t lim = 0xFF00FF00u ^ (seed & 0x00FF00FFu);
  for (int i = 0; i < iters; i++) {
#pragma unroll
    for (int r = 0; r < kUnroll; r++) {
#pragma unroll
      for (int c = 0; c < kChains; c++)
        asm volatile("v_pk_add_u16 %0, %0, %1" : "+v"(a[c]) : "v"(b));
#pragma unroll
      for (int c = 0; c < kChains; c++)
        asm volatile("v_pk_min_u16 %0, %0, %1" : "+v"(a[c]) : "v"(lim));
    }
  }
  uint32_t x = 0;
#pragma unroll
  for (int c = 0; c < kChains; c++) x ^= a[c];
  out[tid] = x;
}

__global__ __launch_bounds__(256) void k_copy(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                              int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += stride)
    dst[i] = src[i];
}

int timed(hipEvent_t e0, hipEvent_t e1, float* ms) {
  if (hipEventSynchronize(e1) != hipSuccess) return -1;
  return hipEventElapsedTime(ms, e0, e1) == hipSuccess ? 0 : -1;
}

}  // namespace

extern "C" {

// Integer VALU peak: kind 0 = 32-bit add/min, 1 = packed 16-bit add/min.
// blocks x 256 threads, iters rounds; out: blocks * 256 uint32 of device
// memory (written so the chains stay live).  *ms: kernel time between HIP
// events on the default stream; *ops: lane operations performed.
int peak_valu(int kind, int blocks, int iters, void* out, float* ms, double* ops) {
  if (blocks <= 0 || iters <= 0 || !out || !ms || !ops || (kind != 0 && kind != 1)) return -1;
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return -1;
  (void)hipEventRecord(e0, 0);
  if (kind == 0)
    hipLaunchKernelGGL(k_valu_i32, dim3(blocks), dim3(256), 0, 0, (uint32_t*)out, iters, 12345u);
  else
    hipLaunchKernelGGL(k_valu_pk_u16, dim3(blocks), dim3(256), 0, 0, (uint32_t*)out, iters,
                       12345u);
  (void)hipEventRecord(e1, 0);
  int st = hipGetLastError() == hipSuccess ? timed(e0, e1, ms) : -1;
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  *ops = (double)blocks * 256.0 * iters * kUnroll * kChains * 2 * (kind == 1 ? 2 : 1);
  return st;
}

// HBM stream: copy bytes (a multiple of 16) from src to dst; *ms as above.
int peak_copy(const void* src, void* dst, int64_t bytes, int blocks, float* ms) {
  if (!src || !dst || bytes <= 0 || bytes % 16 || blocks <= 0 || !ms) return -1;
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return -1;
  (void)hipEventRecord(e0, 0);
  hipLaunchKernelGGL(k_copy, dim3(blocks), dim3(256), 0, 0, (const uint4*)src, (uint4*)dst,
                     bytes / 16);
  (void)hipEventRecord(e1, 0);
  int st = hipGetLastError() == hipSuccess ? timed(e0, e1, ms) : -1;
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  return st;
}

}  // extern "C"
