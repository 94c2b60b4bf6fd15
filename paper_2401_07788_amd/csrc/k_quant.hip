// k_quant.hip -- uniform b-bit min-max quantization (Sec. 2.2 of the paper),
// optionally wrapped in error feedback (Sec. 2.4), and its decompression.
//
// Per group (a sample or a token row): lo = min, hi = max (a -0 reads as +0),
//   code = min(rint((v - lo) / (hi - lo) * (2^b - 1)), 2^b - 1),
//   meta = (lo, (hi - lo) / (2^b - 1)),
// codes packed LSB-first into little-endian 32-bit words; the receiver
// rebuilds lo + code * scale.  b = 32 sends the binary32 values themselves.
// A group is spread over P workgroups that exchange their partial min / max
// through per-workgroup slots and one cross-workgroup barrier; the group's
// values stay in registers between the reduction and the encode.
#include <algorithm>
#include <type_traits>

#include "tc_internal.hpp"
#include "tc_select.hpp"

namespace tc {

constexpr int QVPT = 32;   // elements per thread: 32 * b bits is a whole number of words

__host__ __device__ constexpr uint64_t quant_group_mem_words(uint32_t P) { return 64u + 2u * P; }

template <int B>
__device__ __forceinline__ void pack_codes(const uint32_t (&c)[QVPT], uint32_t (&w)[QVPT * B / 32]) {
#pragma unroll
  for (int j = 0; j < QVPT * B / 32; ++j) w[j] = 0u;
#pragma unroll
  for (int i = 0; i < QVPT; ++i) {
    const int bit = i * B;
    w[bit >> 5] |= c[i] << (bit & 31);
    if ((bit & 31) + B > 32) w[(bit >> 5) + 1] |= c[i] >> (32 - (bit & 31));
  }
}

template <int B>
__device__ __forceinline__ void unpack_codes(const uint32_t (&w)[QVPT * B / 32], uint32_t (&c)[QVPT]) {
  constexpr uint32_t M = (1u << B) - 1u;
#pragma unroll
  for (int i = 0; i < QVPT; ++i) {
    const int bit = i * B;
    uint32_t x = w[bit >> 5] >> (bit & 31);
    if ((bit & 31) + B > 32) x |= w[(bit >> 5) + 1] << (32 - (bit & 31));
    c[i] = x & M;
  }
}

// The code of v in a group with minimum lo and range hi - lo > 0:
// min(rint((v - lo) / range * LV), LV) with the division correctly rounded.
// For range in [2^-125, 2^125] the quotient is first taken as
// (v - lo) * RN(1 / range).  The t = quotient * LV of that form and of the
// direct one differ by at most five roundings of 2^-24 relative each; with
// (v - lo) <= range, t <= 255, so the two lie within 2^-13 of each other and
// round to the same integer unless t is within 2^-10 of a half-integer.
// Those values, and ranges outside the interval, take the division.
template <uint32_t LV>
struct MinMaxCode {
  float lo, range, rcp;
  bool fast;
  __device__ __forceinline__ MinMaxCode(float lo_, float range_) : lo(lo_), range(range_) {
    fast = range >= 0x1p-125f && range <= 0x1p125f;
    rcp = 1.0f / range;
  }
  __device__ __forceinline__ uint32_t operator()(float v) const {
    const float n = v - lo;
    if (fast) {
      const float u = n * rcp;
      const float t = u * (float)LV;
      const float r = rintf(t);
      if (fabsf(t - r) < 0.5f - 0x1p-10f) return min((uint32_t)r, LV);
    }
    const float u = n / range;
    const float t = u * (float)LV;
    return min((uint32_t)rintf(t), LV);
  }
};

// Sender.  Loads, the residual and binary32 codes (b = 32) go in pieces of
// QPE consecutive elements, lanes consecutive, so that every wavefront
// instruction covers contiguous memory; piece j of thread t is element
// (j * NT + t) * QPE of the workgroup's chunk.  Codes of b < 32 bits are
// staged in LDS (one byte per element) and packed by thread t for chunk
// elements [QVPT t, QVPT t + QVPT): QVPT b bits are a whole number of words
// for every b.
constexpr int QPE = 4;                 // elements per piece
constexpr int QNP = QVPT / QPE;        // pieces per thread

template <typename InT, typename OutT, int B, bool EF, int NT>
__global__ __launch_bounds__(NT) void k_quant_pack(QuantArgs a) {
  using R = typename Elem<InT>::raw;
  constexpr int WPT = QVPT * B / 32;   // code words of one packing run (b < 32)
  constexpr uint64_t CH = (uint64_t)NT * QVPT;
  __shared__ float mm[2 * (NT / WAVE)];
  __shared__ uint32_t s_codes[(B == 32) ? 1 : NT * QNP];   // 4 code bytes per word, one word per piece

  const uint32_t P = a.P;
  const uint32_t group = blockIdx.x / P, part = blockIdx.x % P;
  const uint32_t n_groups = gridDim.x / P;
  uint32_t* bar = nullptr;
  uint32_t* slots = nullptr;
  if (P > 1) {
    bar = a.ws + (uint64_t)group * quant_group_mem_words(P);
    slots = bar + 64;
  }
  const uint64_t base = (uint64_t)part * CH;   // the chunk's first element in its group
  auto piece_at = [&](int j) -> uint64_t { return base + ((uint64_t)j * NT + threadIdx.x) * QPE; };
  auto piece_n = [&](int j) -> int { return (int)min((uint64_t)QPE, sat_sub(a.G, piece_at(j))); };

  for (uint64_t grp = group; grp < a.n_grp; grp += n_groups) {
    const uint64_t goff = grp * a.G;
    float v[QVPT];
#pragma unroll
    for (int j = 0; j < QNP; ++j) {
      const int n = piece_n(j);
      R xr[QPE];
      float er[QPE];
      if (n > 0) {
        load_run_partial<R, QPE, true>((const R*)a.x + goff + piece_at(j), n, R{}, xr);
        if constexpr (EF) load_run_partial<float, QPE, true>(a.e + goff + piece_at(j), n, 0.0f, er);
      }
#pragma unroll
      for (int i = 0; i < QPE; ++i) {
        float t = 0.0f;
        if (i < n) {
          t = Elem<InT>::up(xr[i]);
          if constexpr (EF) t = t + er[i];
        }
        v[j * QPE + i] = t;
      }
    }

    float lo = 0.0f, scale = 0.0f;
    if constexpr (B == 32) {
#pragma unroll
      for (int j = 0; j < QNP; ++j) {
        const int n = piece_n(j);
        uint32_t w[QPE];
#pragma unroll
        for (int i = 0; i < QPE; ++i) w[i] = __float_as_uint(v[j * QPE + i]);
        if (n > 0) store_run_partial<uint32_t, QPE, false>(a.codes + grp * a.wpg + piece_at(j), n, w);
        if constexpr (EF) {
#pragma unroll
          for (int i = 0; i < QPE; ++i) v[j * QPE + i] = v[j * QPE + i] - through<OutT>(v[j * QPE + i]);
        }
      }
    } else {
      // ---- min / max of the group
      lo = __int_as_float(0x7F800000);    // +inf
      float hi = __int_as_float(0xFF800000);  // -inf
#pragma unroll
      for (int j = 0; j < QNP; ++j) {
        const int n = piece_n(j);
#pragma unroll
        for (int i = 0; i < QPE; ++i)
          if (i < n) { lo = fminf(lo, v[j * QPE + i]); hi = fmaxf(hi, v[j * QPE + i]); }
      }
      block_minmax<NT>(lo, hi, mm);
      if (P > 1) {
        if (threadIdx.x == 0) {
          st_agent(&slots[2 * part], __float_as_uint(lo));
          st_agent(&slots[2 * part + 1], __float_as_uint(hi));
        }
        group_barrier(bar, P);
        lo = __uint_as_float(ld_agent(&slots[0]));
        hi = __uint_as_float(ld_agent(&slots[1]));
        for (uint32_t j = 1; j < P; ++j) {
          lo = fminf(lo, __uint_as_float(ld_agent(&slots[2 * j])));
          hi = fmaxf(hi, __uint_as_float(ld_agent(&slots[2 * j + 1])));
        }
        // no workgroup may overwrite its slot for the next group before all
        // have read this one
        group_barrier(bar, P);
      }
      lo = lo + 0.0f;   // -0 reads as +0
      hi = hi + 0.0f;
      constexpr uint32_t LV = (1u << B) - 1u;
      const bool flat = (hi == lo);
      const float range = hi - lo;
      scale = flat ? 0.0f : range / (float)LV;
      const MinMaxCode<LV> code_of(lo, flat ? 1.0f : range);
#pragma unroll
      for (int j = 0; j < QNP; ++j) {
        const int n = piece_n(j);
        uint32_t word = 0u;
#pragma unroll
        for (int i = 0; i < QPE; ++i) {
          uint32_t c = 0u;
          if (!flat) c = code_of(v[j * QPE + i]);
          if (i >= n) c = 0u;
          word |= c << (8 * i);
          if constexpr (EF) {
            const float prod = (float)c * scale;
            const float xh = lo + prod;
            v[j * QPE + i] = v[j * QPE + i] - through<OutT>(xh);   // the residual, in place
          }
        }
        s_codes[j * NT + threadIdx.x] = word;
      }
      __syncthreads();
      // ---- pack: thread t takes chunk elements [QVPT t, QVPT t + QVPT)
      uint32_t c[QVPT];
#pragma unroll
      for (int q = 0; q < QVPT / 4; ++q) {
        const uint32_t word = s_codes[threadIdx.x * (QVPT / 4) + q];
#pragma unroll
        for (int i = 0; i < 4; ++i) c[4 * q + i] = (word >> (8 * i)) & 0xFFu;
      }
      __syncthreads();   // the words are rewritten for the next group
      uint32_t w[WPT];
      pack_codes<B>(c, w);
      const uint64_t wo = ((base + (uint64_t)threadIdx.x * QVPT) * (uint64_t)B) / 32u;
      const int nw = (int)min((uint64_t)WPT, sat_sub(a.wpg, wo));
      if (nw > 0) store_run_partial<uint32_t, WPT, false>(a.codes + grp * a.wpg + wo, nw, w);
    }
    if (part == 0 && threadIdx.x == 0) {
      a.meta[2 * grp] = lo;
      a.meta[2 * grp + 1] = scale;
    }
    if constexpr (EF) {
#pragma unroll
      for (int j = 0; j < QNP; ++j) {
        const int n = piece_n(j);
        float r[QPE];
#pragma unroll
        for (int i = 0; i < QPE; ++i) r[i] = v[j * QPE + i];
        if (n > 0) store_run_partial<float, QPE, true>(a.e + goff + piece_at(j), n, r);
      }
    }
  }
  if (P > 1) group_exit<NT>(bar, P, slots, 2ull * P);
}

// Receiver: thread = one run of QVPT consecutive elements of one group; a
// workgroup iteration takes NT consecutive runs over all groups, so short
// groups (token rows) share a workgroup instead of leaving most of its
// threads idle.
template <typename OutT, int B, int NT>
__global__ __launch_bounds__(NT) void k_quant_unpack(UnpackArgs a) {
  using R = typename Elem<OutT>::raw;
  constexpr int WPT = (B == 32) ? QVPT : QVPT * B / 32;
  const uint64_t rpg = (a.G + QVPT - 1) / QVPT;        // runs per group
  const uint64_t n_runs = a.n_grp * rpg;
  for (uint64_t run = (uint64_t)blockIdx.x * NT + threadIdx.x; run < n_runs; run += (uint64_t)gridDim.x * NT) {
    const uint64_t grp = run / rpg;
    const uint64_t c0 = (run % rpg) * QVPT;
    const int nv = (int)min((uint64_t)QVPT, a.G - c0);
    const uint64_t wo = (B == 32) ? c0 : (c0 * (uint64_t)B) / 32u;
    const int nw = (int)min((uint64_t)WPT, sat_sub(a.wpg, wo));
    uint32_t w[WPT];
    load_run_partial<uint32_t, WPT, false>(a.codes + grp * a.wpg + wo, nw, 0u, w);
    R y[QVPT];
    if constexpr (B == 32) {
#pragma unroll
      for (int i = 0; i < QVPT; ++i) y[i] = Elem<OutT>::down(__uint_as_float(w[i]));
    } else {
      const float lo = a.meta[2 * grp], scale = a.meta[2 * grp + 1];
      uint32_t c[QVPT];
      unpack_codes<B>(w, c);
#pragma unroll
      for (int i = 0; i < QVPT; ++i) {
        const float prod = (float)c[i] * scale;
        y[i] = Elem<OutT>::down(lo + prod);
      }
    }
    store_run_partial<R, QVPT, false>((R*)a.y + grp * a.G + c0, nv, y);
  }
}

// The same receiver in pieces of one 16-byte store each (4 binary32 or 8
// 16-bit outputs), lanes consecutive, for the bit widths whose piece codes
// fill whole bytes (b = 2, 4, 8, 32): every load and store instruction of a
// wavefront then covers contiguous memory.  Needs G a multiple of the piece
// and 16-byte aligned arrays (the launcher checks).  One piece per thread:
// more pieces per thread in flight measured slower (fewer workgroups).
template <int BYTES>
__device__ __forceinline__ void load_piece_codes(const uint8_t* p, uint32_t (&w)[(BYTES + 3) / 4]) {
  if constexpr (BYTES == 1) w[0] = *p;
  else if constexpr (BYTES == 2) w[0] = *reinterpret_cast<const uint16_t*>(p);
  else if constexpr (BYTES == 4) w[0] = *reinterpret_cast<const uint32_t*>(p);
  else if constexpr (BYTES == 8) {
    const u32x2 v = *reinterpret_cast<const u32x2*>(p);
    w[0] = v[0]; w[1] = v[1];
  } else {
#pragma unroll
    for (int h = 0; h < BYTES / 16; ++h) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(p + 16 * h);
#pragma unroll
      for (int i = 0; i < 4; ++i) w[4 * h + i] = v[i];
    }
  }
}

template <typename OutT, int B, int NT>
__global__ __launch_bounds__(NT) void k_quant_unpack_pc(UnpackArgs a) {
  using R = typename Elem<OutT>::raw;
  constexpr int PE = 16 / (int)sizeof(R);               // elements per piece
  constexpr int CB = PE * B / 8;                        // code bytes per piece
  const uint64_t ppg = a.G / PE;                        // pieces per group
  const uint64_t n_pieces = a.n_grp * ppg;
  for (uint64_t q = (uint64_t)blockIdx.x * NT + threadIdx.x; q < n_pieces; q += (uint64_t)gridDim.x * NT) {
    const uint64_t grp = q / ppg, p = q - grp * ppg;
    uint32_t c[(CB + 3) / 4];
    load_piece_codes<CB>(reinterpret_cast<const uint8_t*>(a.codes + grp * a.wpg) + p * (uint64_t)CB, c);
    R y[PE];
    if constexpr (B == 32) {
#pragma unroll
      for (int i = 0; i < PE; ++i) y[i] = Elem<OutT>::down(__uint_as_float(c[i]));
    } else {
      const float lo = a.meta[2 * grp], scale = a.meta[2 * grp + 1];
#pragma unroll
      for (int i = 0; i < PE; ++i) {
        const uint32_t code = (c[(i * B) / 32] >> ((i * B) % 32)) & ((1u << B) - 1u);
        const float prod = (float)code * scale;
        y[i] = Elem<OutT>::down(lo + prod);
      }
    }
    store_run<R, PE, true>((R*)a.y + q * PE, y);
  }
}

// ------------------------------------------------------------------ plans
namespace {

constexpr int BIG_NT = 512;
constexpr int ROW_NT = 64;

template <typename InT, typename OutT, bool EF, int NT>
const void* pack_ptr_b(uint32_t b) {
  switch (b) {
    case 1: return (const void*)k_quant_pack<InT, OutT, 1, EF, NT>;
    case 2: return (const void*)k_quant_pack<InT, OutT, 2, EF, NT>;
    case 3: return (const void*)k_quant_pack<InT, OutT, 3, EF, NT>;
    case 4: return (const void*)k_quant_pack<InT, OutT, 4, EF, NT>;
    case 5: return (const void*)k_quant_pack<InT, OutT, 5, EF, NT>;
    case 6: return (const void*)k_quant_pack<InT, OutT, 6, EF, NT>;
    case 7: return (const void*)k_quant_pack<InT, OutT, 7, EF, NT>;
    case 8: return (const void*)k_quant_pack<InT, OutT, 8, EF, NT>;
    case 32: return (const void*)k_quant_pack<InT, OutT, 32, EF, NT>;
  }
  return nullptr;
}

template <typename InT>
const void* pack_ptr(uint32_t b, bool ef, int nt) {
  // the receiver's output dtype is the input dtype
  if (nt == ROW_NT) return ef ? pack_ptr_b<InT, InT, true, ROW_NT>(b) : pack_ptr_b<InT, InT, false, ROW_NT>(b);
  return ef ? pack_ptr_b<InT, InT, true, BIG_NT>(b) : pack_ptr_b<InT, InT, false, BIG_NT>(b);
}

const void* pick_pack(int dt, uint32_t b, bool ef, int nt) {
  if (dt == DT_F32) return pack_ptr<float>(b, ef, nt);
  if (dt == DT_BF16) return pack_ptr<bf16_t>(b, ef, nt);
  return pack_ptr<f16_t>(b, ef, nt);
}

template <typename OutT>
const void* unpack_ptr(uint32_t b) {
  switch (b) {
    case 1: return (const void*)k_quant_unpack<OutT, 1, 256>;
    case 2: return (const void*)k_quant_unpack<OutT, 2, 256>;
    case 3: return (const void*)k_quant_unpack<OutT, 3, 256>;
    case 4: return (const void*)k_quant_unpack<OutT, 4, 256>;
    case 5: return (const void*)k_quant_unpack<OutT, 5, 256>;
    case 6: return (const void*)k_quant_unpack<OutT, 6, 256>;
    case 7: return (const void*)k_quant_unpack<OutT, 7, 256>;
    case 8: return (const void*)k_quant_unpack<OutT, 8, 256>;
    case 32: return (const void*)k_quant_unpack<OutT, 32, 256>;
  }
  return nullptr;
}

}  // namespace

SegPlan plan_quant(int dt, uint32_t bits, bool ef, uint64_t n_grp, uint64_t G) {
  SegPlan p;
  const uint32_t cus = (uint32_t)device_cus();
  p.vpt = QVPT;
  p.nt = (G <= (uint64_t)ROW_NT * QVPT) ? ROW_NT : BIG_NT;
  const uint64_t CH = (uint64_t)p.nt * QVPT;
  p.P = (uint32_t)((G + CH - 1) / CH);
  int occ = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, pick_pack(dt, bits, ef, p.nt), p.nt, 0) != hipSuccess ||
      occ < 1)
    occ = 1;
  const uint64_t cap = (uint64_t)occ * cus;
  p.capacity = cap;
  const uint64_t groups = std::min<uint64_t>(n_grp, std::max<uint64_t>(1, cap / p.P));
  p.n_groups = (uint32_t)groups;
  p.grid = (uint32_t)(groups * p.P);
  const uint64_t ws_groups = std::min<uint64_t>(n_grp, std::max<uint64_t>(1, (uint64_t)cus * 32 / p.P));
  p.ws_words = (p.P > 1) ? ws_groups * quant_group_mem_words(p.P) : 0;
  return p;
}

hipError_t launch_quant(int dt, int out_dt, uint32_t bits, bool ef, const SegPlan& plan, const QuantArgs& args,
                        hipStream_t st) {
  if (out_dt != dt) return hipErrorInvalidValue;
  const void* fn = pick_pack(dt, bits, ef, plan.nt);
  if (!fn) return hipErrorInvalidValue;
  QuantArgs a = args;
  a.P = plan.P;
  void* params[] = {&a};
  return hipLaunchKernel(fn, dim3(plan.grid), dim3(plan.nt), params, 0, st);
}

template <typename OutT>
const void* unpack_pc_ptr(uint32_t b) {
  switch (b) {
    case 2: return (const void*)k_quant_unpack_pc<OutT, 2, 256>;
    case 4: return (const void*)k_quant_unpack_pc<OutT, 4, 256>;
    case 8: return (const void*)k_quant_unpack_pc<OutT, 8, 256>;
    case 32: return (const void*)k_quant_unpack_pc<OutT, 32, 256>;
  }
  return nullptr;
}

hipError_t launch_unpack(int out_dt, uint32_t bits, const UnpackArgs& args, hipStream_t st) {
  // whole 16-byte pieces: whole-byte codes, groups of whole pieces, aligned
  // arrays, and every group's codes aligned to a piece's code load (up to 16
  // bytes)
  const uint64_t pe = 16 / dt_size(out_dt);
  const uint64_t cb = pe * bits / 8;
  const bool pieces = (bits == 2 || bits == 4 || bits == 8 || bits == 32) && (args.G % pe) == 0 &&
                      (((uintptr_t)args.y | (uintptr_t)args.codes) & 15u) == 0 &&
                      ((args.wpg * 4) % std::min<uint64_t>(cb, 16)) == 0;
  if (pieces) {
    const void* f = (out_dt == DT_F32) ? unpack_pc_ptr<float>(bits)
                  : (out_dt == DT_BF16) ? unpack_pc_ptr<bf16_t>(bits) : unpack_pc_ptr<f16_t>(bits);
    const uint64_t n_pieces = args.n_grp * (args.G / pe);
    const uint64_t work = (n_pieces + 255) / 256;   // workgroups of 256 pieces
    const uint64_t grid = std::max<uint64_t>(1, std::min<uint64_t>(work, (uint64_t)device_cus() * 16));
    UnpackArgs a = args;
    void* params[] = {&a};
    return hipLaunchKernel(f, dim3((uint32_t)grid), dim3(256), params, 0, st);
  }
  const void* fn = (out_dt == DT_F32) ? unpack_ptr<float>(bits)
                 : (out_dt == DT_BF16) ? unpack_ptr<bf16_t>(bits) : unpack_ptr<f16_t>(bits);
  if (!fn) return hipErrorInvalidValue;
  const uint64_t runs = args.n_grp * ((args.G + QVPT - 1) / QVPT);
  const uint64_t work = (runs + 255) / 256;   // workgroups of 256 runs
  const uint64_t grid = std::max<uint64_t>(1, std::min<uint64_t>(work, (uint64_t)device_cus() * 8));
  UnpackArgs a = args;
  void* params[] = {&a};
  return hipLaunchKernel(fn, dim3((uint32_t)grid), dim3(256), params, 0, st);
}

TC_DEFINE_ERROR_READER(errors_quant)

}  // namespace tc
