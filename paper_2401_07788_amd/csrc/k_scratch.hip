// k_scratch.hip -- the library-owned scratch of the allocation-free entry
// point (tc_aqsgd_step_noalloc).
//
// The group engine keeps its cross-workgroup counters and exchange records in
// a workspace that must be zero on entry and that every completed call leaves
// zero.  Callers that cannot allocate (code under graph capture, tight serving
// loops) get it from this file-scope device array instead.  Each device that
// loads the library holds its own copy, at its own address, until the process
// ends.  In host code the array's name is only a stand-in for that address:
// the address is looked up once per device with hipGetSymbolAddress and only
// the looked-up pointer is ever handed to a kernel.
#include <mutex>

#include "tc_internal.hpp"

namespace tc {

static __device__ __align__(256) uint32_t scratch[NOALLOC_SCRATCH_BYTES / 4];

namespace {

constexpr int ZERO_NT = 256;
constexpr uint32_t ZERO_GRID = 512;

__global__ __launch_bounds__(ZERO_NT) void k_scratch_zero(uint4* p, uint64_t n16) {
  const uint4 z = make_uint4(0u, 0u, 0u, 0u);
  for (uint64_t i = blockIdx.x * (uint64_t)ZERO_NT + threadIdx.x; i < n16; i += (uint64_t)gridDim.x * ZERO_NT)
    p[i] = z;
}

constexpr int MAX_DEV = 64;
std::mutex g_mu;
void* g_ptr[MAX_DEV] = {};

hipError_t zero(void* p, hipStream_t st) {
  static_assert(NOALLOC_SCRATCH_BYTES % 16 == 0, "whole 16-byte stores");
  hipLaunchKernelGGL(k_scratch_zero, dim3(ZERO_GRID), dim3(ZERO_NT), 0, st, (uint4*)p,
                     (uint64_t)NOALLOC_SCRATCH_BYTES / 16u);
  return hipGetLastError();
}

}  // namespace

// The current device's scratch address.  The first call on a device looks it
// up and enqueues a clearing kernel on `st` (the loader's initial contents are
// not relied on); later calls return the cached address.
hipError_t noalloc_scratch(void** ptr, hipStream_t st) {
  *ptr = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEV) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || ((uintptr_t)p & 255u) != 0) return hipErrorInvalidSymbol;
    e = zero(p, st);
    if (e != hipSuccess) return e;
    g_ptr[dev] = p;
  }
  *ptr = g_ptr[dev];
  return hipSuccess;
}

// After a cross-workgroup wait gave up, the scratch of the current device is
// no longer zero: clear it again (synchronously) if it was set up.
hipError_t noalloc_scratch_reset() {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEV) return hipSuccess;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) return hipSuccess;
  e = zero(g_ptr[dev], nullptr);
  if (e != hipSuccess) return e;
  return hipDeviceSynchronize();
}

}  // namespace tc
