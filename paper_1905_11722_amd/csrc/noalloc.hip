// rc_solve_dual_noalloc: the memory-indexed solve of rc_solve_dual for
// callers that cannot allocate device memory (code under HIP graph capture,
// tight serving loops, harnesses that forbid hipMalloc).  Its table, status
// block and schedule buffers live in one file-scope device array, `scratch`,
// of kNoallocScratchBytes; every GPU the library runs on holds its own copy
// of the array, at its own address, until the process ends.
//
// Host code never passes the array's name to a kernel (on the host it is a
// stand-in, not a device address): the first call on a device, with that
// device current, looks the device address up with hipGetSymbolAddress and
// keeps it per device; every launch then takes that pointer.
//
// All calls on one GPU share that GPU's array, which keeps the last call's
// contents; the table and status are initialised by the solve's own first
// kernel, so nothing needs clearing.  Calls that overlap on one GPU (from
// different threads or streams) race on the array.
#include <hip/hip_runtime.h>

#include <mutex>

#include "rc_internal.h"

namespace rcdp {
namespace {

constexpr size_t kNoallocScratchBytes = (size_t)16 << 20;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// Device address of this device's scratch array (looked up once per device).
int scratch_ptr(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    set_last_error_msg("rc_solve_dual_noalloc: no current HIP device");
    return RC_E_DEVICE;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      set_last_error("hipGetSymbolAddress(scratch)", e);
      return RC_E_DEVICE;
    }
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return RC_OK;
}

size_t round_up(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace
}  // namespace rcdp

using namespace rcdp;

extern "C" int rc_solve_dual_noalloc(rc_family f, int64_t B, int32_t objective, void* stream,
                                     int64_t* t_opt, int64_t* m_opt, int32_t* k,
                                     int32_t* chain_host, int32_t* seg_host, uint8_t* cached_host,
                                     int64_t* overhead, int64_t* peak, int64_t* cache_mem) {
  DualBuffers b;
  const int st = dual_buffers(f, B, objective, &b);
  if (st != RC_OK) return st;
  const size_t n = (size_t)f->g->n;
  const size_t o_st = 0;
  const size_t o_chain = o_st + round_up(sizeof(DevStatus));
  const size_t o_seg = o_chain + round_up(sizeof(int32_t) * (size_t)f->F);
  const size_t o_cached = o_seg + round_up(sizeof(int32_t) * n);
  const size_t o_D = o_cached + round_up(n);
  const size_t total = o_D + sizeof(uint32_t) * (size_t)b.cells;
  if (total > kNoallocScratchBytes) {
    set_last_error_msg("rc_solve_dual_noalloc: the table needs more than the 16 MiB scratch");
    return RC_E_SCRATCH;
  }
  void* base = nullptr;
  const int sp = scratch_ptr(&base);
  if (sp != RC_OK) return sp;
  unsigned char* p = static_cast<unsigned char*>(base);
  b.st = reinterpret_cast<DevStatus*>(p + o_st);
  b.chain = reinterpret_cast<int32_t*>(p + o_chain);
  b.seg = reinterpret_cast<int32_t*>(p + o_seg);
  b.cached = p + o_cached;
  b.D = reinterpret_cast<uint32_t*>(p + o_D);
  return dual_solve(f, objective, b, nullptr, nullptr, reinterpret_cast<hipStream_t>(stream),
                    t_opt, m_opt, k, chain_host, seg_host, cached_host, overhead, peak, cache_mem);
}
