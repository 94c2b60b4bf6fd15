// k_global.hip -- TopK over a segment too long to stay on chip (a whole
// micro-batch of a large language model, Sec. 3.2-scale activations), with
// error feedback (Sec. 2.4) and, optionally, the kept list quantized as one
// min-max group (Sec. 2.2).
//
// A chain of kernels on one stream; kernel boundaries are the global syncs:
//   hist<1>, pick<1>   12-bit digit of all keys        -> bin b1
//   hist<2>, pick<2>   next 12 bits of keys in b1       -> bin b2
//   hist<3>, pick<3>   last 7 bits of keys in (b1, b2)  -> threshold T, ties r
//   emit               one ordered pass over 4096-element tiles: counts,
//                      decoupled look-back for the tile's payload offset,
//                      compaction of idx (and values), the dense residual,
//                      the block table, min / max of the kept values
//   qpack (quantized kept list only)  codes of the kept list, meta, and the
//                      residual at the kept entries (X read back from e,
//                      where emit left it)
//   clean              tile states and counters back to zero
// The input is read four times (three histogram passes and the emit pass).
#include <algorithm>

#include "tc_internal.hpp"
#include "tc_select.hpp"

namespace tc {

constexpr int G_NT = 256;
constexpr int G_VPT = 16;
constexpr uint64_t G_TILE = (uint64_t)G_NT * G_VPT;   // == BLOCK_LEN
static_assert(G_TILE == BLOCK_LEN, "one emit tile per block of the block table");

// state words (workspace)
enum : int {
  ST_B1 = 0, ST_NEED2, ST_B2, ST_NEED3, ST_T, ST_R,
  ST_TICKET, ST_EXIT, ST_MIN, ST_MAX,     // emit bookkeeping; ST_MIN/MAX hold ordered keys
  ST_WORDS = 64
};

__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_order_key(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}

template <typename InT, bool EF>
__device__ __forceinline__ void load_tile_values(const GlobalArgs& a, uint64_t t0, int nv, float (&v)[G_VPT]) {
  using R = typename Elem<InT>::raw;
  R xr[G_VPT];
  if (nv > 0) load_run_partial<R, G_VPT, true>((const R*)a.x + t0, nv, R{}, xr);
  if constexpr (EF) {
    float er[G_VPT];
    if (nv > 0) load_run_partial<float, G_VPT, true>(a.e + t0, nv, 0.0f, er);
#pragma unroll
    for (int i = 0; i < G_VPT; ++i) v[i] = (i < nv) ? Elem<InT>::up(xr[i]) + er[i] : 0.0f;
  } else {
#pragma unroll
    for (int i = 0; i < G_VPT; ++i) v[i] = (i < nv) ? Elem<InT>::up(xr[i]) : 0.0f;
  }
}

// ------------------------------------------------------------- histograms
template <typename InT, bool EF, int PASS>
__global__ __launch_bounds__(G_NT) void k_g_hist(GlobalArgs a) {
  constexpr int NB = (PASS == 3) ? LAST_BINS : HIST_BINS;
  __shared__ uint32_t hist[NB];
  for (int b = threadIdx.x; b < NB; b += G_NT) hist[b] = 0u;
  __syncthreads();
  const uint32_t* st = a.state;
  const uint32_t b1 = (PASS >= 2) ? st[ST_B1] : 0u;
  const uint32_t p24 = (PASS == 3) ? ((st[ST_B1] << 12) | st[ST_B2]) : 0u;
  uint32_t zc = 0;
  for (uint64_t tile = blockIdx.x; tile < a.n_tiles; tile += gridDim.x) {
    const uint64_t t0 = tile * G_TILE + (uint64_t)threadIdx.x * G_VPT;
    const int nv = (int)min((uint64_t)G_VPT, sat_sub(a.L, t0));
    float v[G_VPT];
    load_tile_values<InT, EF>(a, t0, nv, v);
#pragma unroll
    for (int i = 0; i < G_VPT; ++i) {
      if (i < nv) {
        const uint32_t kk = mag_key(v[i]);
        bool in;
        uint32_t d;
        if constexpr (PASS == 1) { in = true; d = kk >> 19; }
        else if constexpr (PASS == 2) { in = (kk >> 19) == b1; d = (kk >> 7) & 0xFFFu; }
        else { in = (kk >> 7) == p24; d = kk & 0x7Fu; }
        if (in) {
          if (kk == 0u) ++zc;
          else atomicAdd(&hist[d], 1u);
        }
      }
    }
  }
  const uint32_t zs = wave_sum(zc);
  if (lane_id() == 0 && zs) atomicAdd(&hist[0], zs);
  __syncthreads();
  uint32_t* gh = a.hist + (PASS - 1) * HIST_BINS;
  for (int b = threadIdx.x; b < NB; b += G_NT)
    if (hist[b]) add_agent(&gh[b], hist[b]);
}

// one workgroup: find the bin of this pass, advance the state, clear the
// histogram for the next call
template <int PASS>
__global__ __launch_bounds__(512) void k_g_pick(GlobalArgs a) {
  constexpr int NB = (PASS == 3) ? LAST_BINS : HIST_BINS;
  __shared__ uint32_t h[NB];
  __shared__ uint32_t scratch[512 / WAVE + 2];
  __shared__ uint32_t found[2];
  uint32_t* gh = a.hist + (PASS - 1) * HIST_BINS;
  for (int b = threadIdx.x; b < NB; b += 512) { h[b] = ld_agent(&gh[b]); st_agent(&gh[b], 0u); }
  __syncthreads();
  uint32_t* st = a.state;
  const uint32_t need = (PASS == 1) ? (uint32_t)a.k : (PASS == 2) ? st[ST_NEED2] : st[ST_NEED3];
  find_bin<512, NB>(h, need, scratch, found);
  if (threadIdx.x == 0) {
    if constexpr (PASS == 1) { st[ST_B1] = found[0]; st[ST_NEED2] = need - found[1]; }
    else if constexpr (PASS == 2) { st[ST_B2] = found[0]; st[ST_NEED3] = need - found[1]; }
    else {
      st[ST_T] = (((st[ST_B1] << 12) | st[ST_B2]) << 7) | found[0];
      st[ST_R] = need - found[1];
    }
  }
}

// ------------------------------------------------------------------- emit
// Tile state word: bit 63..62 flag (1 = own counts, 2 = inclusive prefix),
// bits 61..31 keys > T, bits 30..0 keys == T.
constexpr uint64_t TF_AGG = 1ull << 62, TF_INC = 2ull << 62, TF_MASK = 3ull << 62;
__device__ __forceinline__ uint64_t tile_word(uint64_t flag, uint32_t gt, uint32_t eq) {
  return flag | ((uint64_t)gt << 31) | (uint64_t)eq;
}
constexpr uint32_t LOOKBACK_SPIN_LIMIT = 1u << 22;

template <typename InT, bool EF, bool QKEPT>
__global__ __launch_bounds__(G_NT) void k_g_emit(GlobalArgs a) {
  using R = typename Elem<InT>::raw;
  __shared__ uint32_t s_tile;
  __shared__ uint32_t scratch[G_NT / WAVE + 2];
  __shared__ uint32_t s_prefix[2];
  __shared__ float s_mm[2 * (G_NT / WAVE)];
  uint64_t* tiles = reinterpret_cast<uint64_t*>(a.tiles);
  uint32_t* st = a.state;
  const uint32_t T = (a.k == 0) ? 0xFFFFFFFFu : st[ST_T];
  const uint32_t r = (a.k == 0) ? 0u : st[ST_R];
  float kmin = __builtin_inff(), kmax = -__builtin_inff();
  for (;;) {
    if (threadIdx.x == 0) s_tile = __hip_atomic_fetch_add(&st[ST_TICKET], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const uint64_t tile = s_tile;
    __syncthreads();
    if (tile >= a.n_tiles) break;
    const uint64_t t0 = tile * G_TILE + (uint64_t)threadIdx.x * G_VPT;
    const int nv = (int)min((uint64_t)G_VPT, sat_sub(a.L, t0));
    float v[G_VPT];
    load_tile_values<InT, EF>(a, t0, nv, v);
    uint32_t key[G_VPT];
#pragma unroll
    for (int i = 0; i < G_VPT; ++i) key[i] = mag_key(v[i]);
    uint32_t gt = 0, eq = 0;
#pragma unroll
    for (int i = 0; i < G_VPT; ++i)
      if (i < nv) { gt += key[i] > T; eq += key[i] == T; }
    uint32_t tot;
    const uint32_t ex = block_excl_scan<G_NT>(gt | (eq << 16), scratch, tot);
    const uint32_t gt_t = tot & 0xFFFFu, eq_t = tot >> 16;
    // ---- the tile's offset: publish own counts, look back over predecessors
    if (threadIdx.x == 0) {
      uint32_t pg = 0, pe = 0;
      if (tile == 0) {
        __hip_atomic_store(&tiles[0], tile_word(TF_INC, gt_t, eq_t), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      } else {
        __hip_atomic_store(&tiles[tile], tile_word(TF_AGG, gt_t, eq_t), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        uint64_t j = tile - 1;
        uint32_t spins = 0;
        for (;;) {
          const uint64_t w = __hip_atomic_load(&tiles[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          const uint64_t f = w & TF_MASK;
          if (f == 0) {
            __builtin_amdgcn_s_sleep(1);
            if (++spins > LOOKBACK_SPIN_LIMIT) { raise_error(KERR_TIMEOUT); break; }
            continue;
          }
          pg += (uint32_t)((w >> 31) & 0x7FFFFFFFu);
          pe += (uint32_t)(w & 0x7FFFFFFFu);
          if (f == TF_INC || j == 0) break;
          --j;
        }
        __builtin_amdgcn_s_waitcnt(0);
        __hip_atomic_store(&tiles[tile], tile_word(TF_INC, pg + gt_t, pe + eq_t), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      }
      s_prefix[0] = pg;
      s_prefix[1] = pe;
    }
    __syncthreads();
    const uint32_t gt_before = s_prefix[0], eq_before = s_prefix[1];
    // ---- placement inside the tile (ties: the lowest indices overall)
    const uint32_t quota_t = min(sat_sub(r, eq_before), eq_t);
    const uint32_t gt_ex = ex & 0xFFFFu, eq_ex = ex >> 16;
    const uint32_t tile_first = gt_before + min(eq_before, r);
    uint32_t pos = tile_first + gt_ex + min(eq_ex, quota_t);
    const uint32_t tie_keep = min(sat_sub(quota_t, eq_ex), (uint32_t)G_VPT);
    uint32_t ties = 0;
    float eo[G_VPT];
#pragma unroll
    for (int i = 0; i < G_VPT; ++i) {
      bool kept = false;
      if (i < nv) {
        const bool tie = key[i] == T;
        kept = key[i] > T || (tie && ties < tie_keep);
        ties += tie ? 1u : 0u;
        if (kept) {
          if (pos < a.k) {
            a.idx[pos] = (uint32_t)(t0 + i);
            if constexpr (!QKEPT) ((R*)a.val)[pos] = Elem<InT>::down(v[i]);
          } else {
            raise_error(KERR_INTERNAL);
          }
          ++pos;
          if constexpr (QKEPT) { kmin = fminf(kmin, v[i]); kmax = fmaxf(kmax, v[i]); }
        }
      }
      if constexpr (EF) {
        // the quantized case corrects the kept entries later (qpack reads X back from here)
        eo[i] = (kept && !QKEPT) ? v[i] - through<InT>(v[i]) : v[i] - 0.0f;
      }
    }
    if constexpr (EF) {
      if (nv > 0) store_run_partial<float, G_VPT, true>(a.e + t0, nv, eo);
    }
    if (a.blk && threadIdx.x == 0) a.blk[tile] = tile_first;
  }
  if (a.blk && blockIdx.x == 0 && threadIdx.x == 0) a.blk[a.n_tiles] = (uint32_t)a.k;
  if constexpr (QKEPT) {
    block_minmax<G_NT>(kmin, kmax, s_mm);
    if (threadIdx.x == 0 && kmin <= kmax) {
      __hip_atomic_fetch_min(&st[ST_MIN], order_key(kmin), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_fetch_max(&st[ST_MAX], order_key(kmax), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// ------------------------------------------------------------------ qpack
// codes of the kept list (one min-max group), meta, and with error feedback
// the residual at the kept entries: e[idx_j] holds X there (emit left it)
constexpr int QP_VPT = 32;

template <int B, typename OutT, bool EF>
__global__ __launch_bounds__(G_NT) void k_g_qpack(GlobalArgs a) {
  constexpr int WPT = (B == 32) ? QP_VPT : QP_VPT * B / 32;
  const uint32_t* st = a.state;
  float lo = 0.0f, scale = 0.0f, hi = 0.0f;
  const bool any = a.k > 0;
  if (any) {
    lo = from_order_key(st[ST_MIN]) + 0.0f;
    hi = from_order_key(st[ST_MAX]) + 0.0f;
  }
  constexpr uint32_t LV = (B == 32) ? 0u : (1u << B) - 1u;
  if (B != 32 && any && hi != lo) scale = (hi - lo) / (float)LV;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    a.meta[0] = (B == 32) ? 0.0f : lo;
    a.meta[1] = scale;
  }
  for (uint64_t j0 = ((uint64_t)blockIdx.x * G_NT + threadIdx.x) * QP_VPT; j0 < a.k;
       j0 += (uint64_t)gridDim.x * G_NT * QP_VPT) {
    const int n = (int)min((uint64_t)QP_VPT, a.k - j0);
    uint32_t ix[QP_VPT];
    float x[QP_VPT];
#pragma unroll
    for (int i = 0; i < QP_VPT; ++i) {
      ix[i] = (i < n) ? a.idx[j0 + i] : 0u;
      x[i] = (i < n && ix[i] < a.L) ? a.e[ix[i]] : 0.0f;
    }
    uint32_t w[WPT];
    uint32_t c[QP_VPT];
    if constexpr (B == 32) {
#pragma unroll
      for (int i = 0; i < QP_VPT; ++i) w[i] = __float_as_uint(x[i]);
    } else {
      const float range = hi - lo;
#pragma unroll
      for (int i = 0; i < QP_VPT; ++i) {
        uint32_t q = 0;
        if (hi != lo) {
          const float u = (x[i] - lo) / range;
          const float t = u * (float)LV;
          q = min((uint32_t)rintf(t), LV);
        }
        c[i] = (i < n) ? q : 0u;
      }
#pragma unroll
      for (int q = 0; q < WPT; ++q) w[q] = 0u;
#pragma unroll
      for (int i = 0; i < QP_VPT; ++i) {
        const int bit = i * B;
        w[bit >> 5] |= c[i] << (bit & 31);
        if ((bit & 31) + B > 32) w[(bit >> 5) + 1] |= c[i] >> (32 - (bit & 31));
      }
    }
    const uint64_t wo = (B == 32) ? j0 : (j0 * (uint64_t)B) / 32u;
    const int nw = (int)min((uint64_t)WPT, sat_sub(a.wpg, wo));
    if (nw > 0) store_run_partial<uint32_t, WPT, true>(a.codes + wo, nw, w);
    if constexpr (EF) {
#pragma unroll
      for (int i = 0; i < QP_VPT; ++i) {
        if (i < n) {
          if (ix[i] >= a.L) { raise_error(KERR_INTERNAL); continue; }
          float rec;
          if constexpr (B == 32) rec = x[i];
          else { const float prod = (float)c[i] * scale; rec = lo + prod; }
          a.e[ix[i]] = x[i] - through<OutT>(rec);
        }
      }
    }
  }
}

// back to the zero-filled workspace: tile states, counters and the state words
__global__ __launch_bounds__(G_NT) void k_g_clean(GlobalArgs a) {
  for (uint64_t i = (uint64_t)blockIdx.x * G_NT + threadIdx.x; i < 2 * a.n_tiles; i += (uint64_t)gridDim.x * G_NT)
    st_agent(&a.tiles[i], 0u);
  if (blockIdx.x == 0)
    for (int i = threadIdx.x; i < ST_WORDS; i += G_NT) st_agent(&a.state[i], 0u);
}

// min/max start values before emit
__global__ void k_g_minmax_init(GlobalArgs a) {
  if (threadIdx.x == 0) {
    a.state[ST_MIN] = 0xFFFFFFFFu;
    a.state[ST_MAX] = 0u;
    a.state[ST_TICKET] = 0u;
  }
}

// ------------------------------------------------------------------ plans
namespace {

template <typename InT, bool EF>
const void* hist_ptr(int pass) {
  if (pass == 1) return (const void*)k_g_hist<InT, EF, 1>;
  if (pass == 2) return (const void*)k_g_hist<InT, EF, 2>;
  return (const void*)k_g_hist<InT, EF, 3>;
}
template <typename InT>
const void* hist_ptr_ef(bool ef, int pass) { return ef ? hist_ptr<InT, true>(pass) : hist_ptr<InT, false>(pass); }
const void* pick_hist(int dt, bool ef, int pass) {
  if (dt == DT_F32) return hist_ptr_ef<float>(ef, pass);
  if (dt == DT_BF16) return hist_ptr_ef<bf16_t>(ef, pass);
  return hist_ptr_ef<f16_t>(ef, pass);
}

template <typename InT>
const void* emit_ptr(bool ef, bool qkept) {
  if (ef) return qkept ? (const void*)k_g_emit<InT, true, true> : (const void*)k_g_emit<InT, true, false>;
  return qkept ? (const void*)k_g_emit<InT, false, true> : (const void*)k_g_emit<InT, false, false>;
}
const void* pick_emit(int dt, bool ef, bool qkept) {
  if (dt == DT_F32) return emit_ptr<float>(ef, qkept);
  if (dt == DT_BF16) return emit_ptr<bf16_t>(ef, qkept);
  return emit_ptr<f16_t>(ef, qkept);
}

template <typename OutT, bool EF>
const void* qpack_ptr_b(uint32_t b) {
  switch (b) {
    case 1: return (const void*)k_g_qpack<1, OutT, EF>;
    case 2: return (const void*)k_g_qpack<2, OutT, EF>;
    case 3: return (const void*)k_g_qpack<3, OutT, EF>;
    case 4: return (const void*)k_g_qpack<4, OutT, EF>;
    case 5: return (const void*)k_g_qpack<5, OutT, EF>;
    case 6: return (const void*)k_g_qpack<6, OutT, EF>;
    case 7: return (const void*)k_g_qpack<7, OutT, EF>;
    case 8: return (const void*)k_g_qpack<8, OutT, EF>;
    case 32: return (const void*)k_g_qpack<32, OutT, EF>;
  }
  return nullptr;
}
const void* pick_qpack(int out_dt, bool ef, uint32_t b) {
  if (out_dt == DT_F32) return ef ? qpack_ptr_b<float, true>(b) : qpack_ptr_b<float, false>(b);
  if (out_dt == DT_BF16) return ef ? qpack_ptr_b<bf16_t, true>(b) : qpack_ptr_b<bf16_t, false>(b);
  return ef ? qpack_ptr_b<f16_t, true>(b) : qpack_ptr_b<f16_t, false>(b);
}

hipError_t launch(const void* fn, uint32_t grid, uint32_t nt, const GlobalArgs& args, hipStream_t st) {
  if (!fn) return hipErrorInvalidValue;
  GlobalArgs a = args;
  void* params[] = {&a};
  return hipLaunchKernel(fn, dim3(grid), dim3(nt), params, 0, st);
}

}  // namespace

uint64_t global_ws_words(uint64_t L) {
  // state, three histograms, and two words per tile
  return (uint64_t)ST_WORDS + 3ull * HIST_BINS + 2ull * n_blocks(L);
}

void global_ws_carve(uint32_t* ws, uint64_t L, GlobalArgs& a) {
  a.state = ws;
  a.hist = ws + ST_WORDS;
  a.tiles = ws + ST_WORDS + 3 * HIST_BINS;
  a.n_tiles = n_blocks(L);
}

hipError_t launch_global(int dt, bool ef, uint32_t qbits, const GlobalArgs& args, hipStream_t st) {
  // the quantized kept list reads X back from the residual buffer
  if (qbits != 0 && !ef) return hipErrorInvalidValue;
  const uint32_t cus = (uint32_t)device_cus();
  const uint32_t grid = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(args.n_tiles, (uint64_t)cus * 8));
  const bool qkept = qbits != 0;
  hipError_t e = hipSuccess;
  if (args.k > 0) {
    for (int pass = 1; pass <= 3 && e == hipSuccess; ++pass) {
      e = launch(pick_hist(dt, ef, pass), grid, G_NT, args, st);
      if (e == hipSuccess) {
        const void* pk = (pass == 1) ? (const void*)k_g_pick<1> : (pass == 2) ? (const void*)k_g_pick<2>
                                                                                : (const void*)k_g_pick<3>;
        e = launch(pk, 1, 512, args, st);
      }
    }
  }
  if (e == hipSuccess) e = launch((const void*)k_g_minmax_init, 1, 64, args, st);
  if (e == hipSuccess) e = launch(pick_emit(dt, ef, qkept), grid, G_NT, args, st);
  if (e == hipSuccess && qkept) {
    const uint64_t work = (args.k + (uint64_t)G_NT * QP_VPT - 1) / ((uint64_t)G_NT * QP_VPT);
    const uint32_t qgrid = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(work, (uint64_t)cus * 8));
    e = launch(pick_qpack(dt, ef, qbits), qgrid, G_NT, args, st);
  }
  if (e == hipSuccess) e = launch((const void*)k_g_clean, std::min<uint32_t>(grid, 256), G_NT, args, st);
  return e;
}

TC_DEFINE_ERROR_READER(errors_global)

}  // namespace tc
