// k_check.hip -- precondition checks of the debug build of libtc (TC_DEBUG).
//
// The release library assumes what the paper's operations need to be
// well defined and does not spend bandwidth on checking it: finite inputs
// (Sec. 2.2's hi - lo, Sec. 2.4's x + e), and, for AQ-SGD (Sec. 2.5), a
// change a - m[id] and an updated buffer value that fit the buffer's dtype.
// The debug build runs these kernels before the real launch and returns
// TC_ERR_PRECONDITION when one of them reports a violation, with nothing else
// enqueued.  Each check ORs a bit into a per-device word that the host reads
// after synchronising the stream.
#include <algorithm>

#include "tc_device.hpp"
#include "tc_internal.hpp"

namespace tc {

static __device__ uint32_t g_check_flags;

constexpr int CHK_NT = 256;
constexpr uint32_t CHK_GRID = 1024;

// |v| at most half the binary32 maximum: then hi - lo of any group is finite
__device__ __forceinline__ bool fits_range(float v) { return fabsf(v) <= 1.7014117e38f; }

template <typename T>
__global__ __launch_bounds__(CHK_NT) void k_check_values(const typename Elem<T>::raw* x, const float* e, uint64_t n) {
  uint32_t bad = 0;
  for (uint64_t i = blockIdx.x * (uint64_t)CHK_NT + threadIdx.x; i < n; i += (uint64_t)gridDim.x * CHK_NT) {
    const float v = Elem<T>::up(x[i]);
    if (!isfinite(v)) bad |= CHK_NONFINITE;
    if (e) {
      const float s = v + e[i];
      if (!isfinite(e[i]) || !isfinite(s)) bad |= CHK_NONFINITE;
      else if (!fits_range(s)) bad |= CHK_RANGE;
    } else if (isfinite(v) && !fits_range(v)) {
      bad |= CHK_RANGE;
    }
  }
  if (bad) __hip_atomic_fetch_or(&g_check_flags, bad, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// AQ-SGD: a and the rows m[id] finite, the change d = a - m and the updated
// value m + wire(d) finite after rounding to T.  Rows with an id out of range
// are left to the kernels' own reporting.
template <typename T>
__global__ __launch_bounds__(CHK_NT) void k_check_aqsgd(const typename Elem<T>::raw* a,
                                                        const typename Elem<T>::raw* m, const int64_t* ids,
                                                        uint64_t n_ids, uint64_t L, uint64_t n_samples) {
  using Raw = typename Elem<T>::raw;
  uint32_t bad = 0;
  const uint64_t n = n_ids * L;
  for (uint64_t i = blockIdx.x * (uint64_t)CHK_NT + threadIdx.x; i < n; i += (uint64_t)gridDim.x * CHK_NT) {
    const uint64_t b = i / L, j = i - b * L;
    const int64_t id = ids[b];
    if (id < 0 || (uint64_t)id >= n_samples) continue;
    const float av = Elem<T>::up(a[i]);
    const float mv = Elem<T>::up(m[(uint64_t)id * L + j]);
    if (!isfinite(av) || !isfinite(mv)) { bad |= CHK_NONFINITE; continue; }
    const Raw w = Elem<T>::down(av - mv);
    const float wv = Elem<T>::up(w);
    if (!isfinite(wv) || !isfinite(Elem<T>::up(Elem<T>::down(mv + wv)))) bad |= CHK_RANGE;
  }
  if (bad) __hip_atomic_fetch_or(&g_check_flags, bad, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

namespace {
uint32_t grid_for(uint64_t n) {
  const uint64_t g = (n + CHK_NT - 1) / CHK_NT;
  return (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(g, CHK_GRID));
}

hipError_t read_flags(hipStream_t st, uint32_t* flags) {
  hipError_t e = hipStreamSynchronize(st);
  if (e != hipSuccess) return e;
  uint32_t v = 0;
  e = hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_check_flags), sizeof(v), 0, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return e;
  *flags = v;
  if (v) {
    const uint32_t z = 0;
    e = hipMemcpyToSymbol(HIP_SYMBOL(g_check_flags), &z, sizeof(z), 0, hipMemcpyHostToDevice);
  }
  return e;
}
}  // namespace

hipError_t check_values(int dt, const void* x, const float* e, uint64_t n, hipStream_t st, uint32_t* flags) {
  *flags = 0;
  if (n == 0) return hipSuccess;
  const dim3 g(grid_for(n)), b(CHK_NT);
  if (dt == DT_F32) hipLaunchKernelGGL(k_check_values<float>, g, b, 0, st, (const float*)x, e, n);
  else if (dt == DT_BF16) hipLaunchKernelGGL(k_check_values<bf16_t>, g, b, 0, st, (const uint16_t*)x, e, n);
  else hipLaunchKernelGGL(k_check_values<f16_t>, g, b, 0, st, (const uint16_t*)x, e, n);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  return read_flags(st, flags);
}

hipError_t check_aqsgd(int dt, const void* a, const void* m, const int64_t* ids, uint64_t n_ids, uint64_t L,
                       uint64_t n_samples, hipStream_t st, uint32_t* flags) {
  *flags = 0;
  if (n_ids * L == 0) return hipSuccess;
  const dim3 g(grid_for(n_ids * L)), b(CHK_NT);
  if (dt == DT_F32)
    hipLaunchKernelGGL(k_check_aqsgd<float>, g, b, 0, st, (const float*)a, (const float*)m, ids, n_ids, L, n_samples);
  else if (dt == DT_BF16)
    hipLaunchKernelGGL(k_check_aqsgd<bf16_t>, g, b, 0, st, (const uint16_t*)a, (const uint16_t*)m, ids, n_ids, L,
                       n_samples);
  else
    hipLaunchKernelGGL(k_check_aqsgd<f16_t>, g, b, 0, st, (const uint16_t*)a, (const uint16_t*)m, ids, n_ids, L,
                       n_samples);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  return read_flags(st, flags);
}

}  // namespace tc
