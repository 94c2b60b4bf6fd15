// tc_device.hpp -- device-side building blocks for the gfx950 boundary
// compressors: element formats, vector memory access, wave64 / workgroup
// reductions and scans, and the bounded cross-workgroup barrier.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tc {

constexpr int WAVE = 64;

// kernel-side error bits, OR-ed into a per-device sticky word
enum : uint32_t {
  KERR_TIMEOUT = 1u,     // a cross-workgroup wait gave up (co-residency violated)
  KERR_BAD_ID = 2u,      // an AQ-SGD sample id outside [0, n_samples)
  KERR_BAD_INDEX = 4u,   // a payload index outside its segment or chunk
  KERR_INTERNAL = 8u,    // a selection placed an entry past k (never expected)
};

// one word per kernel translation unit (internal linkage); the host reads
// it through hipMemcpyFromSymbol in that same unit
static __device__ uint32_t g_kernel_errors;

__device__ __forceinline__ void raise_error(uint32_t bits) {
  __hip_atomic_fetch_or(&g_kernel_errors, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------------ formats
// Element types: float, and 16-bit patterns tagged by these wrappers so that
// templates can tell bfloat16 from binary16.
struct bf16_t { uint16_t u; };
struct f16_t { uint16_t u; };

template <typename T> struct Elem;
template <> struct Elem<float> {
  using raw = float;
  static __device__ __forceinline__ float up(float v) { return v; }
  static __device__ __forceinline__ float down(float v) { return v; }
};
template <> struct Elem<bf16_t> {
  using raw = uint16_t;
  // exact: bfloat16 is the high half of a binary32
  static __device__ __forceinline__ float up(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }
  // round to nearest even (hardware conversion, default rounding mode)
  static __device__ __forceinline__ uint16_t down(float v) {
    return __builtin_bit_cast(uint16_t, (__bf16)v);
  }
};
template <> struct Elem<f16_t> {
  using raw = uint16_t;
  static __device__ __forceinline__ float up(uint16_t h) {
    return (float)__builtin_bit_cast(_Float16, h);
  }
  static __device__ __forceinline__ uint16_t down(float v) {
    return __builtin_bit_cast(uint16_t, (_Float16)v);
  }
};

// the value a receiver holds after v went through element type T
template <typename T>
__device__ __forceinline__ float through(float v) { return Elem<T>::up(Elem<T>::down(v)); }

// magnitude key: the binary32 pattern without its sign.  For finite values
// the unsigned order of keys is the order of |v|, and +0 / -0 share key 0.
__device__ __forceinline__ uint32_t mag_key(float v) { return __float_as_uint(v) & 0x7FFFFFFFu; }

// Tells the optimiser that register-resident values may have changed (no
// instruction is emitted).  Called between the phases that each derive keys
// from the same values, it makes every phase recompute what it needs instead
// of keeping another phase's derived values alive across barriers, which
// would exhaust the registers.
template <int R, int E>
__device__ __forceinline__ void refresh(float (&v)[R][E]) {
#pragma unroll
  for (int j = 0; j < R; ++j)
#pragma unroll
    for (int i = 0; i < E; ++i) asm volatile("" : "+v"(v[j][i]));
}

// ------------------------------------------------------------ vector access
// Load/store N consecutive raw elements starting at p (element units).
// Uses 16-byte accesses when the run is 16-byte aligned and a multiple of 16
// bytes, else 8-byte, else scalar accesses.  STREAM marks data touched once
// per launch (the boundary tensors): those accesses carry the non-temporal
// hint so that they do not displace reused lines.  Loads and stores take the
// hint only where one instruction of a wavefront covers whole 128-byte lines
// (lane-contiguous 16-byte accesses, copy_lds_to_global).  A thread's run of
// several 16-byte accesses covers each line only across instructions: with
// the hint, loads then fetch a line more than once and stores write it out
// piecewise (measured: up to 1.8x the bytes), while cached loads and write-
// back stores let the L2 serve and merge the pieces.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <bool STREAM, typename V>
__device__ __forceinline__ V vload(const V* p) {
  if constexpr (STREAM) return __builtin_nontemporal_load(p);
  else return *p;
}
template <bool STREAM, typename V>
__device__ __forceinline__ void vstore(V* p, V v) {
  if constexpr (STREAM) __builtin_nontemporal_store(v, p);
  else *p = v;
}

// A read at an address that is the same for the whole wavefront, of memory
// that no kernel in flight writes, in the constant address space: the scalar
// unit serves it, counted apart from the vector loads, so that waiting for
// it does not wait for them.
template <typename T>
__device__ __forceinline__ T load_uniform(const T* p) {
  return *(const __attribute__((address_space(4))) T*)p;
}

template <typename R, int N, bool STREAM = false>
__device__ __forceinline__ void load_run(const R* __restrict__ p, R (&out)[N]) {
  constexpr int BYTES = N * (int)sizeof(R);
  const uintptr_t a = (uintptr_t)p;
  if constexpr (BYTES % 16 == 0) {
    if ((a & 15u) == 0) {
      constexpr int PER = 16 / (int)sizeof(R);
#pragma unroll
      for (int i = 0; i < N / PER; ++i) {
        const u32x4 w = vload<STREAM>(reinterpret_cast<const u32x4*>(p + i * PER));
        __builtin_memcpy(&out[i * PER], &w, 16);
      }
      return;
    }
  }
  if constexpr (BYTES % 8 == 0) {
    if ((a & 7u) == 0) {
      constexpr int PER = 8 / (int)sizeof(R);
#pragma unroll
      for (int i = 0; i < N / PER; ++i) {
        const u32x2 w = vload<STREAM>(reinterpret_cast<const u32x2*>(p + i * PER));
        __builtin_memcpy(&out[i * PER], &w, 8);
      }
      return;
    }
  }
#pragma unroll
  for (int i = 0; i < N; ++i) out[i] = p[i];
}

template <typename R, int N, bool STREAM = false>
__device__ __forceinline__ void store_run(R* __restrict__ p, const R (&in)[N]) {
  constexpr int BYTES = N * (int)sizeof(R);
  const uintptr_t a = (uintptr_t)p;
  if constexpr (BYTES % 16 == 0) {
    if ((a & 15u) == 0) {
      constexpr int PER = 16 / (int)sizeof(R);
#pragma unroll
      for (int i = 0; i < N / PER; ++i) {
        u32x4 w;
        __builtin_memcpy(&w, &in[i * PER], 16);
        vstore<STREAM>(reinterpret_cast<u32x4*>(p + i * PER), w);
      }
      return;
    }
  }
  if constexpr (BYTES % 8 == 0) {
    if ((a & 7u) == 0) {
      constexpr int PER = 8 / (int)sizeof(R);
#pragma unroll
      for (int i = 0; i < N / PER; ++i) {
        u32x2 w;
        __builtin_memcpy(&w, &in[i * PER], 8);
        vstore<STREAM>(reinterpret_cast<u32x2*>(p + i * PER), w);
      }
      return;
    }
  }
#pragma unroll
  for (int i = 0; i < N; ++i) p[i] = in[i];
}

// one 4-element piece (16 bytes of fp32, 8 of a 16-bit format), which the
// caller has aligned: no alignment test
template <typename Raw, bool STREAM>
__device__ __forceinline__ void load_piece(const Raw* p, Raw (&out)[4]) {
  if constexpr (sizeof(Raw) == 4) {
    const u32x4 w = vload<STREAM>(reinterpret_cast<const u32x4*>(p));
    __builtin_memcpy(out, &w, 16);
  } else {
    const u32x2 w = vload<STREAM>(reinterpret_cast<const u32x2*>(p));
    __builtin_memcpy(out, &w, 8);
  }
}

// Load a run that may be cut short at `n` valid elements (n <= N); elements
// past n are left as `fill`.
template <typename R, int N, bool STREAM = false>
__device__ __forceinline__ void load_run_partial(const R* __restrict__ p, int n, R fill, R (&out)[N]) {
  if (n >= N) { load_run<R, N, STREAM>(p, out); return; }
#pragma unroll
  for (int i = 0; i < N; ++i) out[i] = (i < n) ? p[i] : fill;
}

template <typename R, int N, bool STREAM = false>
__device__ __forceinline__ void store_run_partial(R* __restrict__ p, int n, const R (&in)[N]) {
  if (n >= N) { store_run<R, N, STREAM>(p, in); return; }
#pragma unroll
  for (int i = 0; i < N; ++i)
    if (i < n) p[i] = in[i];
}

// Copy n consecutive elements from LDS to device memory, all threads of the
// workgroup together: unaligned head and tail element by element, the body
// in 16-byte stores at 16-byte aligned addresses.
template <int NT, typename R>
__device__ __forceinline__ void copy_lds_to_global(R* __restrict__ dst, const R* src, uint32_t n) {
  constexpr uint32_t PER = 16 / sizeof(R);
  const uint32_t mis = (uint32_t)(((uintptr_t)dst / sizeof(R)) % PER);
  const uint32_t head = min(n, (PER - mis) % PER);
  const uint32_t body = (n - head) / PER;
  const int t = (int)threadIdx.x;
  if ((uint32_t)t < head) dst[t] = src[t];
  if ((((uintptr_t)(src + head)) & 15u) == 0) {
    // source pieces 16-byte aligned as well: one LDS read each
    const u32x4* s4 = reinterpret_cast<const u32x4*>(src + head);
    for (uint32_t q = (uint32_t)t; q < body; q += NT) vstore<true>(reinterpret_cast<u32x4*>(dst + head + q * PER), s4[q]);
  } else {
    for (uint32_t q = (uint32_t)t; q < body; q += NT) {
      R tmp[PER];
#pragma unroll
      for (uint32_t i = 0; i < PER; ++i) tmp[i] = src[head + q * PER + i];
      u32x4 w;
      __builtin_memcpy(&w, tmp, 16);
      vstore<true>(reinterpret_cast<u32x4*>(dst + head + q * PER), w);
    }
  }
  const uint32_t done = head + body * PER;
  if ((uint32_t)t < n - done) dst[done + t] = src[done + t];
}

// 0/1 comparisons of 31-bit keys as integer arithmetic on bit fields: the
// per-element loops then keep their flags in vector registers (no 64-bit
// lane masks, which exhaust the scalar registers in long unrolled loops).
__device__ __forceinline__ uint32_t gt31(uint32_t a, uint32_t b) {   // a > b, both < 2^31
  return __builtin_amdgcn_ubfe(b - a, 31, 1);
}
__device__ __forceinline__ uint32_t eq31(uint32_t a, uint32_t b) {   // a == b, both < 2^31
  const uint32_t x = a ^ b;
  return __builtin_amdgcn_ubfe((x - 1u) & ~x, 31, 1);
}
// f ? x : y with f in {0, 1}
__device__ __forceinline__ uint32_t pick(uint32_t f, uint32_t x, uint32_t y) { return ((x ^ y) & (0u - f)) ^ y; }

// a - b clamped at 0, written without a guarded subtraction.  The device
// compiler of this toolchain can turn `b < a ? a - b : 0` into an unguarded
// no-wrap subtraction and then use the implied a >= b to fold unrelated
// min() calls away; every clamped difference in this library goes through
// this form instead.
template <typename T>
__device__ __forceinline__ T sat_sub(T a, T b) { return a - min(a, b); }

// --------------------------------------------------------- wave64 helpers
__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (WAVE - 1)); }

// Cross-lane steps use DPP (data-parallel primitives: lane shifts inside a
// 16-lane row, then row broadcasts), which run on the VALU without an LDS
// round trip.  Lanes without a source lane read `old`.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t old, uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)x, CTRL, ROW_MASK, 0xF, false);
}
constexpr int DPP_ROW_SHR1 = 0x111, DPP_ROW_SHR2 = 0x112, DPP_ROW_SHR4 = 0x114, DPP_ROW_SHR8 = 0x118;
constexpr int DPP_ROW_BCAST15 = 0x142, DPP_ROW_BCAST31 = 0x143;

// inclusive prefix sum over the 64 lanes (all lanes must be active)
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  x += dpp_u32<DPP_ROW_SHR1, 0xF>(0u, x);
  x += dpp_u32<DPP_ROW_SHR2, 0xF>(0u, x);
  x += dpp_u32<DPP_ROW_SHR4, 0xF>(0u, x);
  x += dpp_u32<DPP_ROW_SHR8, 0xF>(0u, x);
  x += dpp_u32<DPP_ROW_BCAST15, 0xA>(0u, x);   // rows 1, 3 add the end of rows 0, 2
  x += dpp_u32<DPP_ROW_BCAST31, 0xC>(0u, x);   // rows 2, 3 add the end of row 1
  return x;
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(x), WAVE - 1);
}

// running min / max in the same lane pattern; lane 63 ends with the result
template <bool MAX>
__device__ __forceinline__ float wave_minmax(float x) {
  const uint32_t id = __float_as_uint(MAX ? -__builtin_inff() : __builtin_inff());
  auto op = [](float a, float b) { return MAX ? fmaxf(a, b) : fminf(a, b); };
  uint32_t u = __float_as_uint(x);
  u = __float_as_uint(op(__uint_as_float(u), __uint_as_float(dpp_u32<DPP_ROW_SHR1, 0xF>(id, u))));
  u = __float_as_uint(op(__uint_as_float(u), __uint_as_float(dpp_u32<DPP_ROW_SHR2, 0xF>(id, u))));
  u = __float_as_uint(op(__uint_as_float(u), __uint_as_float(dpp_u32<DPP_ROW_SHR4, 0xF>(id, u))));
  u = __float_as_uint(op(__uint_as_float(u), __uint_as_float(dpp_u32<DPP_ROW_SHR8, 0xF>(id, u))));
  u = __float_as_uint(op(__uint_as_float(u), __uint_as_float(dpp_u32<DPP_ROW_BCAST15, 0xA>(id, u))));
  u = __float_as_uint(op(__uint_as_float(u), __uint_as_float(dpp_u32<DPP_ROW_BCAST31, 0xC>(id, u))));
  return __uint_as_float((uint32_t)__builtin_amdgcn_readlane((int)u, WAVE - 1));
}

__device__ __forceinline__ float wave_min(float x) { return wave_minmax<false>(x); }
__device__ __forceinline__ float wave_max(float x) { return wave_minmax<true>(x); }

template <bool MAX>
__device__ __forceinline__ uint32_t wave_uminmax(uint32_t x) {
  const uint32_t id = MAX ? 0u : 0xFFFFFFFFu;
  auto op = [](uint32_t a, uint32_t b) { return MAX ? max(a, b) : min(a, b); };
  x = op(x, dpp_u32<DPP_ROW_SHR1, 0xF>(id, x));
  x = op(x, dpp_u32<DPP_ROW_SHR2, 0xF>(id, x));
  x = op(x, dpp_u32<DPP_ROW_SHR4, 0xF>(id, x));
  x = op(x, dpp_u32<DPP_ROW_SHR8, 0xF>(id, x));
  x = op(x, dpp_u32<DPP_ROW_BCAST15, 0xA>(id, x));
  x = op(x, dpp_u32<DPP_ROW_BCAST31, 0xC>(id, x));
  return (uint32_t)__builtin_amdgcn_readlane((int)x, WAVE - 1);
}

// ------------------------------------------------------- workgroup helpers
// scratch must hold NT/64 + 1 words of LDS.  All threads of the workgroup
// must call these (they contain barriers).  Wave totals go through LDS once;
// every wave then adds the totals of the waves before it itself, so there is
// one LDS round trip between the two barriers and no serial chain.
template <int NT>
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* scratch, uint32_t& total) {
  constexpr int NW = NT / WAVE;
  const int w = (int)threadIdx.x / WAVE;
  uint32_t incl = wave_incl_scan(v);
  if constexpr (NW == 1) {
    total = (uint32_t)__builtin_amdgcn_readlane((int)incl, WAVE - 1);
    return incl - v;
  } else {
    if (lane_id() == WAVE - 1) scratch[w] = incl;
    __syncthreads();
    uint32_t pre = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const uint32_t x = scratch[i];
      pre += (i < w) ? x : 0u;
      tot += x;
    }
    total = tot;
    __syncthreads();
    return pre + incl - v;
  }
}

template <int NT>
__device__ __forceinline__ uint32_t block_sum(uint32_t v, uint32_t* scratch) {
  constexpr int NW = NT / WAVE;
  uint32_t s = wave_sum(v);
  if constexpr (NW == 1) {
    return s;
  } else {
    const int w = (int)threadIdx.x / WAVE;
    if (lane_id() == 0) scratch[w] = s;
    __syncthreads();
    uint32_t t = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) t += scratch[i];
    __syncthreads();
    return t;
  }
}

template <int NT>
__device__ __forceinline__ void block_minmax(float& lo, float& hi, float* scratch /*2*NT/64*/) {
  constexpr int NW = NT / WAVE;
  lo = wave_min(lo);
  hi = wave_max(hi);
  if constexpr (NW > 1) {
    const int w = (int)threadIdx.x / WAVE;
    if (lane_id() == 0) { scratch[w] = lo; scratch[NW + w] = hi; }
    __syncthreads();
    lo = scratch[0];
    hi = scratch[NW];
#pragma unroll
    for (int i = 1; i < NW; ++i) { lo = fminf(lo, scratch[i]); hi = fmaxf(hi, scratch[NW + i]); }
    __syncthreads();
  }
}

// ------------------------------------------------ cross-workgroup barrier
// A sense-reversing barrier among the P workgroups of one group (state[0..2]:
// arrival count, sense, exit count; see group_exit).
//
// Everything one workgroup hands to another inside a launch (histograms,
// slots, these counters) is written and read with device-scope atomics
// (add_agent / st_agent / ld_agent), which are coherent at device scope by
// themselves.  The barrier therefore only has to order them: each wave
// waits until its own memory operations have completed before the
// workgroup arrives, and every later read is issued after the wait has seen
// the flip.  No cache write-back or invalidate is needed (those would only
// matter for plain loads and stores, which never cross workgroups here).
// The wait is bounded: if the other workgroups do not arrive (they are not
// co-resident), it gives up, raises KERR_TIMEOUT and lets the kernel finish.
constexpr uint32_t BARRIER_SPIN_LIMIT = 1u << 19;

__device__ __forceinline__ void group_barrier(uint32_t* state, uint32_t P) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t* count = state;
    uint32_t* sense = state + 1;
    const uint32_t s0 = __hip_atomic_load(sense, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t prev = __hip_atomic_fetch_add(count, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev == P - 1) {
      __hip_atomic_store(count, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __builtin_amdgcn_s_waitcnt(0);
      __hip_atomic_store(sense, s0 ^ 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
      uint32_t spins = 0;
      while (__hip_atomic_load(sense, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == s0) {
        __builtin_amdgcn_s_sleep(1);
        ++spins;
        // once any wait on the device has given up, stop waiting at once
        if ((spins & 1023u) == 0u &&
            (__hip_atomic_load(&g_kernel_errors, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & KERR_TIMEOUT))
          break;
        if (spins > BARRIER_SPIN_LIMIT) { raise_error(KERR_TIMEOUT); break; }
      }
    }
  }
  __syncthreads();
}

// Leave a group's workspace zero-filled: every workgroup counts itself out in
// state[2]; the last one clears `words` (per-workgroup slots, which are
// rewritten before every read and so never cleared in flight), the sense word
// and the counter.  Nobody waits here.
template <int NT>
__device__ __forceinline__ void group_exit(uint32_t* state, uint32_t P, uint32_t* words, uint64_t n_words) {
  __shared__ uint32_t last_out;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t prev = __hip_atomic_fetch_add(state + 2, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    last_out = (prev == P - 1) ? 1u : 0u;
  }
  __syncthreads();
  if (last_out) {
    for (uint64_t i = threadIdx.x; i < n_words; i += NT)
      __hip_atomic_store(words + i, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (threadIdx.x == 0) {
      __hip_atomic_store(state + 1, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(state + 2, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

__device__ __forceinline__ uint32_t ld_agent(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void add_agent(uint32_t* p, uint32_t v) {
  __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_agent64(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// host side: read (and optionally clear) this translation unit's error word
#define TC_DEFINE_ERROR_READER(fn)                                                          \
  hipError_t fn(uint32_t* bits, bool clear) {                                               \
    uint32_t v = 0;                                                                         \
    hipError_t st = hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_kernel_errors), sizeof(v), 0,      \
                                        hipMemcpyDeviceToHost);                             \
    if (st != hipSuccess) return st;                                                        \
    *bits = v;                                                                              \
    if (clear && v) {                                                                       \
      const uint32_t z = 0;                                                                 \
      st = hipMemcpyToSymbol(HIP_SYMBOL(g_kernel_errors), &z, sizeof(z), 0,                 \
                             hipMemcpyHostToDevice);                                        \
    }                                                                                       \
    return st;                                                                              \
  }                                                                                         \
  /* ORs bits into the word from the host (device idle: the caller synchronizes) */         \
  hipError_t fn##_raise(uint32_t bits) {                                                    \
    uint32_t v = 0;                                                                         \
    hipError_t st = hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_kernel_errors), sizeof(v), 0,      \
                                        hipMemcpyDeviceToHost);                             \
    if (st != hipSuccess) return st;                                                        \
    v |= bits;                                                                              \
    return hipMemcpyToSymbol(HIP_SYMBOL(g_kernel_errors), &v, sizeof(v), 0,                 \
                             hipMemcpyHostToDevice);                                        \
  }

}  // namespace tc
