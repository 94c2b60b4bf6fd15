// k_global.hip -- TopK over a segment too long to stay on chip (a whole
// micro-batch of a large language model, Sec. 3.2-scale activations), with
// error feedback (Sec. 2.4) and, optionally, the kept list quantized as one
// min-max group (Sec. 2.2).
//
// A chain of kernels on one stream; kernel boundaries are the global syncs,
// and the last workgroup to finish a kernel takes the decision that kernel
// feeds:
//   sample   histogram of the top 12 key bits over about 512 evenly spaced
//            4096-element tiles -> a band of digits that holds the k-th
//            largest key with high probability
//   band     one pass over all keys: count the keys above the band, write
//            the values inside it to a candidate list (exact check that the
//            band holds the k-th key)
//   pass 1-3 the three radix digits (12/12/7 bits) -> threshold T and the tie
//            quota r, over the candidate list when the band held the k-th
//            key, else over the whole segment; when the band is narrow the
//            band pass counts its digits and pass 1 has nothing left to do
//   tcount   per-tile counts and offsets; (quantized kept list) on the way,
//            the min / max of the kept candidates, so that with the band's
//            values emit can quantize
//   emit     one ordered pass over tiles: kept entries marked, encoded from
//            a compacted list, payload written coalesced, the dense
//            residual, the block table
//   finish   (quantized kept list, only when min / max could not be fixed in
//            advance) codes, meta and the residual at the kept entries; then
//            tile words, candidate list and state back to zero
// The input is read twice on the candidate path (band, emit), plus the
// sample.
//
// Device-scope atomics on one address serialize at the memory side, so
// every counter that all workgroups touch is spread over 8 slots 128 bytes
// apart (workgroup w uses slot w % 8): kernel completion counts, the
// candidate sub-lists and the band's sums.
#include <algorithm>
#include <cmath>
#include <type_traits>

#include "tc_internal.hpp"
#include "tc_select.hpp"

namespace tc {

constexpr int G_NT = 256;
constexpr int G_VPT = 16;
constexpr uint64_t G_TILE = (uint64_t)G_NT * G_VPT;   // == BLOCK_LEN
static_assert(G_TILE == BLOCK_LEN, "one emit tile per block of the block table");
constexpr uint32_t SAMPLE_TILES = 512;      // tiles in the sample (every stride-th tile; all if fewer)
constexpr uint32_t SAMPLE_GRID = 256;
constexpr uint32_t CAND_GRID = 256;         // workgroups that read the candidate list
constexpr uint32_t NSLOT = 8;               // slots of a spread counter
constexpr uint32_t SLOT_WORDS = 32;         // 128 bytes between slots
constexpr uint32_t CBUF = (uint32_t)G_TILE; // band: candidates buffered in LDS

// state words (workspace); every word is zero at rest
enum : int {
  ST_B1 = 0, ST_NEED2, ST_B2, ST_NEED3, ST_T, ST_R,
  ST_MIN, ST_MAX,       // emit: min (as ~order key) / max (order key) of the kept values
  ST_BLO, ST_BHI,       // band of top digits
  ST_ABOVE,             // keys above the band
  ST_FAST,              // 1: the band held the k-th key, passes run on candidates
  ST_NEED1,
  ST_AMIN, ST_AMAX,     // values with key > T (as ST_MIN / ST_MAX)
  ST_TPOS, ST_TNEG,     // candidates with key == T, by sign
  ST_PRE,               // 1: lo / hi / scale known before emit
  ST_LO, ST_HI, ST_SCALE,
  ST_P1,                // 1: the band pass already found the first digit (pass 1 has nothing to do)
  ST_SPREAD = 64,       // spread counters: NSLOT slots + a top word, SLOT_WORDS apart
  SP_WORDS = (NSLOT + 1) * SLOT_WORDS,
  SP_DONE = ST_SPREAD,                  // kernel completion (top word: slots done)
  SP_NCAND = SP_DONE + SP_WORDS,        // candidates per sub-list
  SP_ABOVE = SP_NCAND + SP_WORDS,       // band: keys above the band
  SP_AMIN = SP_ABOVE + SP_WORDS,        // band: values above the band
  SP_AMAX = SP_AMIN + SP_WORDS,
  ST_WORDS = 2048
};
constexpr uint32_t BD_MAX = 32;    // band digits counted per digit in the band pass (narrower bands)
constexpr int SP_BD = SP_AMAX + SP_WORDS;   // [NSLOT][BD_MAX] candidates per band digit
static_assert(SP_BD + NSLOT * BD_MAX <= ST_WORDS, "state words");

__device__ __forceinline__ uint32_t* slot(uint32_t* st, int sp, uint32_t c) { return st + sp + SLOT_WORDS * c; }

// order-preserving map of floats to unsigned (finite values map into
// [0x007FFFFF, 0xFF800000]); the minimum is kept as the maximum of the
// complement, so that 0 means "none" for both
__device__ __forceinline__ uint32_t order_key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_order_key(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}
__device__ __forceinline__ void push_minmax(uint32_t* st, int wmin, int wmax, float lo, float hi) {
  if (lo <= hi) {
    __hip_atomic_fetch_max(&st[wmin], ~order_key(lo), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_fetch_max(&st[wmax], order_key(hi), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// true in every thread of the workgroup that finishes last; it sees every
// device-scope update the other workgroups made before finishing.  Each
// workgroup counts in slot (blockIdx % 8); the last of a slot counts in the
// top word.
// G: the workgroups that take part (blockIdx < G; the whole grid by default).
__device__ __forceinline__ bool last_block(uint32_t* st, uint32_t G = 0u) {
  __shared__ uint32_t s_last;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    if (G == 0u) G = gridDim.x;
    const uint32_t c = blockIdx.x % NSLOT;
    const uint32_t n_c = (G - 1 - c) / NSLOT + 1;   // workgroups of this slot
    const uint32_t n_slots = min(G, NSLOT);
    uint32_t* sc = slot(st, SP_DONE, c);
    uint32_t* top = slot(st, SP_DONE, NSLOT);
    bool last = false;
    if (__hip_atomic_fetch_add(sc, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == n_c - 1) {
      __hip_atomic_store(sc, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __builtin_amdgcn_s_waitcnt(0);
      if (__hip_atomic_fetch_add(top, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == n_slots - 1) {
        __hip_atomic_store(top, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        last = true;
      }
    }
    s_last = last ? 1u : 0u;
  }
  __syncthreads();
  return s_last != 0u;
}

// sum / min / max over the slots of a spread counter
__device__ __forceinline__ uint64_t slot_sum(uint32_t* st, int sp) {
  uint64_t t = 0;
  for (uint32_t c = 0; c < NSLOT; ++c) t += ld_agent(slot(st, sp, c));
  return t;
}
__device__ __forceinline__ uint32_t slot_max(uint32_t* st, int sp) {
  uint32_t t = 0;
  for (uint32_t c = 0; c < NSLOT; ++c) t = max(t, ld_agent(slot(st, sp, c)));
  return t;
}

template <typename InT, bool EF>
__device__ __forceinline__ void load_tile_values(const GlobalArgs& a, uint64_t t0, int nv, float (&v)[G_VPT]) {
  using R = typename Elem<InT>::raw;
  R xr[G_VPT];
  if (nv > 0) load_run_partial<R, G_VPT, false>((const R*)a.x + t0, nv, R{}, xr);
  if constexpr (EF) {
    float er[G_VPT];
    if (nv > 0) load_run_partial<float, G_VPT, false>(a.e + t0, nv, 0.0f, er);
#pragma unroll
    for (int i = 0; i < G_VPT; ++i) v[i] = (i < nv) ? Elem<InT>::up(xr[i]) + er[i] : 0.0f;
  } else {
#pragma unroll
    for (int i = 0; i < G_VPT; ++i) v[i] = (i < nv) ? Elem<InT>::up(xr[i]) : 0.0f;
  }
}

// One thread's 16 elements of a whole tile as loaded (16-byte accesses),
// fetched one tile ahead in the band and emit passes, so that the next
// tile's loads are in flight while this one is worked on.
template <typename InT, bool EF>
struct TileRaw {
  static constexpr int XW = G_VPT * (int)sizeof(typename Elem<InT>::raw) / 16;
  u32x4 x[XW];
  u32x4 e[EF ? G_VPT / 4 : 1];
};
// whole 16-byte runs: both arrays 16-byte aligned
__device__ __forceinline__ bool tiles_prefetchable(const GlobalArgs& a) {
  return (((uintptr_t)a.x | (uintptr_t)a.e) & 15u) == 0;
}
// the tile lies wholly inside the segment
__device__ __forceinline__ bool tile_whole(const GlobalArgs& a, uint64_t tile) {
  return tile < a.n_tiles && (tile + 1) * G_TILE <= a.L;
}
template <typename InT, bool EF>
__device__ __forceinline__ void tile_fetch(const GlobalArgs& a, uint64_t tile, TileRaw<InT, EF>& r) {
  using R = typename Elem<InT>::raw;
  const uint64_t t0 = tile * G_TILE + (uint64_t)threadIdx.x * G_VPT;
  const u32x4* px = reinterpret_cast<const u32x4*>((const R*)a.x + t0);
#pragma unroll
  for (int i = 0; i < TileRaw<InT, EF>::XW; ++i) r.x[i] = px[i];
  if constexpr (EF) {
    const u32x4* pe = reinterpret_cast<const u32x4*>(a.e + t0);
#pragma unroll
    for (int i = 0; i < G_VPT / 4; ++i) r.e[i] = pe[i];
  }
}
template <typename InT, bool EF>
__device__ __forceinline__ void tile_values(const TileRaw<InT, EF>& r, float (&v)[G_VPT]) {
  using R = typename Elem<InT>::raw;
#pragma unroll
  for (int i = 0; i < G_VPT; ++i) {
    float x;
    if constexpr (sizeof(R) == 4) {
      x = __uint_as_float(r.x[i / 4][i % 4]);
    } else {
      const uint32_t w = r.x[i / 8][(i % 8) / 2];
      x = Elem<InT>::up((R)((i & 1) ? (w >> 16) : (w & 0xFFFFu)));
    }
    if constexpr (EF) x = x + __uint_as_float(r.e[i / 4][i % 4]);
    v[i] = x;
  }
}

__device__ __forceinline__ void zero_lds_bins(uint32_t* h, int nb) {
  for (int b = threadIdx.x; b < nb; b += G_NT) h[b] = 0u;
}

// LDS histogram -> the device histogram (non-zero bins only)
__device__ __forceinline__ void merge_bins(const uint32_t* h, uint32_t* gh, int nb) {
  for (int b = threadIdx.x; b < nb; b += G_NT)
    if (h[b]) add_agent(&gh[b], h[b]);
}

// the last workgroup: copy a device histogram into LDS and zero it.  A
// thread's loads all go out before any is used (one round trip, not one per
// bin).
__device__ __forceinline__ void take_bins(uint32_t* h, uint32_t* gh, int nb) {
  constexpr int PER = HIST_BINS / G_NT;
  static_assert(HIST_BINS % G_NT == 0, "whole bins per thread");
  uint32_t v[PER];
#pragma unroll
  for (int r = 0; r < PER; ++r) {
    const int b = (int)threadIdx.x + r * G_NT;
    v[r] = (b < nb) ? ld_agent(&gh[b]) : 0u;
  }
#pragma unroll
  for (int r = 0; r < PER; ++r) {
    const int b = (int)threadIdx.x + r * G_NT;
    if (b < nb) {
      h[b] = v[r];
      st_agent(&gh[b], 0u);
    }
  }
  __syncthreads();
}

// ---------------------------------------------------------------- sample
template <typename InT, bool EF>
__global__ __launch_bounds__(G_NT) void k_g_sample(GlobalArgs a) {
  __shared__ uint32_t hist[HIST_BINS];
  __shared__ uint32_t scratch[G_NT / WAVE + 2];
  __shared__ uint32_t found[2];
  zero_lds_bins(hist, HIST_BINS);
  __syncthreads();
  uint32_t* st = a.state;
  const uint64_t stride = a.sample_stride;
  const uint64_t n_s = (a.n_tiles + stride - 1) / stride;
  uint32_t zc = 0;
  for (uint64_t q = blockIdx.x; q < n_s; q += gridDim.x) {
    const uint64_t t0 = q * stride * G_TILE + (uint64_t)threadIdx.x * G_VPT;
    const int nv = (int)min((uint64_t)G_VPT, sat_sub(a.L, t0));
    float v[G_VPT];
    load_tile_values<InT, EF>(a, t0, nv, v);
#pragma unroll
    for (int i = 0; i < G_VPT; ++i) {
      if (i < nv) {
        const uint32_t kk = mag_key(v[i]);
        if (kk == 0u) ++zc;
        else atomicAdd(&hist[kk >> 19], 1u);
      }
    }
  }
  const uint32_t zs = wave_sum(zc);
  if (lane_id() == 0 && zs) atomicAdd(&hist[0], zs);
  __syncthreads();
  uint32_t* gh = a.hist;   // histogram 0
  merge_bins(hist, gh, HIST_BINS);
  if (!last_block(st)) return;
  take_bins(hist, gh, HIST_BINS);
  uint32_t part = 0;
  for (int b = threadIdx.x; b < HIST_BINS; b += G_NT) part += hist[b];
  const uint32_t ns = block_sum<G_NT>(part, scratch);
  // ranks of the sample that bracket the k-th key of the whole segment:
  // the expected rank +- 4 binomial standard deviations (+16)
  const double p = (double)a.k / (double)a.L;
  const double ks = p * (double)ns;
  const double d = 4.0 * sqrt(ks * (1.0 - p)) + 16.0;
  const double lo_r = fmin(fmax(floor(ks - d), 1.0), (double)ns);
  const double hi_r = fmin(fmax(ceil(ks + d), 1.0), (double)ns);
  find_bin<G_NT, HIST_BINS>(hist, (uint32_t)lo_r, scratch, found);
  const uint32_t bhi = found[0];
  __syncthreads();
  find_bin<G_NT, HIST_BINS>(hist, (uint32_t)hi_r, scratch, found);
  if (threadIdx.x == 0) {
    st[ST_BHI] = bhi;
    st[ST_BLO] = found[0];
  }
}

// ------------------------------------------------------------------- band
// candidate sub-list c holds a.cand_cap / a.n_sub values at a.cand + c * that
__device__ __forceinline__ uint64_t sub_cap(const GlobalArgs& a) { return a.cand_cap / a.n_sub; }

// Tile records (4 words per tile).  band writes [0] keys above the band,
// [1] where the tile's candidates start in the candidate array, [2] how many;
// tcount overwrites [0] keys > T, [1] keys == T, [2] / [3] the exclusive
// prefix of those over the tiles of its workgroup.
constexpr uint32_t TL_MAX = 64;   // band: tiles with buffered candidates before a flush

template <typename InT, bool EF>
__global__ __launch_bounds__(G_NT) void k_g_band(GlobalArgs a) {
  __shared__ uint32_t s_cand[CBUF];
  __shared__ __attribute__((aligned(16))) uint32_t s_vals[G_TILE];   // one tile's values, when it has candidates
  __shared__ uint32_t s_tl_tile[TL_MAX], s_tl_pos[TL_MAX];
  __shared__ uint32_t scratch[G_NT / WAVE + 2];
  __shared__ uint32_t s_base;
  __shared__ float s_mm[2 * (G_NT / WAVE)];
  __shared__ uint32_t s_bd[BD_MAX];   // this workgroup's candidates per band digit
  uint32_t* st = a.state;
  if (threadIdx.x < BD_MAX) s_bd[threadIdx.x] = 0u;
  // the quantized kept list's emit ORs codes into the words it shares with
  // neighbouring tiles: they start at zero
  if (a.codes) {
    const uint64_t gsz = (uint64_t)gridDim.x * G_NT;
    for (uint64_t i = (uint64_t)blockIdx.x * G_NT + threadIdx.x; i < a.wpg; i += gsz) a.codes[i] = 0u;
  }
  const uint32_t blo = st[ST_BLO], bhi = st[ST_BHI];
  const bool count_digits = bhi - blo < BD_MAX;   // the band's digits are counted here
  const uint32_t c = blockIdx.x % a.n_sub;
  const uint64_t capc = sub_cap(a);
  uint32_t nbuf = 0, ntl = 0;   // workgroup-uniform
  // buffered candidates -> the workgroup's sub-list (one reservation), and
  // the buffered tiles' record word [1]
  auto flush = [&]() {
    __syncthreads();
    if (threadIdx.x == 0)
      s_base = __hip_atomic_fetch_add(slot(st, SP_NCAND, c), nbuf, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const uint64_t base = s_base;
    uint32_t* list = a.cand + c * capc;
    for (uint32_t j = threadIdx.x; j < nbuf; j += G_NT)
      if (base + j < capc) list[base + j] = s_cand[j];
    for (uint32_t j = threadIdx.x; j < ntl; j += G_NT)
      a.tiles[4 * (uint64_t)s_tl_tile[j] + 1] = (uint32_t)min(c * capc + base + s_tl_pos[j], a.cand_cap);
    __syncthreads();
    nbuf = 0;
    ntl = 0;
  };
  float amin = __builtin_inff(), amax = -__builtin_inff();
  uint32_t above_all = 0;   // workgroup-uniform
  const bool pf = tiles_prefetchable(a);
  TileRaw<InT, EF> nxt;
  bool have = pf && tile_whole(a, blockIdx.x);
  if (have) tile_fetch<InT, EF>(a, blockIdx.x, nxt);
  for (uint64_t tile = blockIdx.x; tile < a.n_tiles; tile += gridDim.x) {
    const uint64_t t0 = tile * G_TILE + (uint64_t)threadIdx.x * G_VPT;
    const int nv = (int)min((uint64_t)G_VPT, sat_sub(a.L, t0));
    float v[G_VPT];
    if (have) tile_values<InT, EF>(nxt, v);
    else load_tile_values<InT, EF>(a, t0, nv, v);
    have = pf && tile_whole(a, tile + gridDim.x);
    if (have) tile_fetch<InT, EF>(a, tile + gridDim.x, nxt);
    // above the band / inside it, as bit masks (bit i: element i); digits
    // are 12-bit, so the sign bit of a difference compares them
    uint32_t am = 0, bm = 0;
#pragma unroll
    for (int i = 0; i < G_VPT; ++i) {
      const uint32_t dg = mag_key(v[i]) >> 19;
      const uint32_t up = (bhi - dg) >> 31;
      am |= up << i;
      bm |= ((~((dg - blo) | (bhi - dg))) >> 31) << i;
      amin = fminf(amin, up ? v[i] : __builtin_inff());
      amax = fmaxf(amax, up ? v[i] : -__builtin_inff());
    }
    const uint32_t valid = (nv >= G_VPT) ? 0xFFFFu : ((1u << max(nv, 0)) - 1u);
    bm &= valid;
    const uint32_t above = (uint32_t)__builtin_popcount(am & valid), inb = (uint32_t)__builtin_popcount(bm);
    uint32_t tot;
    uint32_t off = block_excl_scan<G_NT>(inb | (above << 16), scratch, tot) & 0xFFFFu;
    const uint32_t n_t = tot & 0xFFFFu, ab_t = tot >> 16;
    above_all += ab_t;
    if (n_t && (nbuf + n_t > CBUF || ntl == TL_MAX)) flush();
    if (threadIdx.x == 0) {
      a.tiles[4 * tile + 0] = ab_t;
      a.tiles[4 * tile + 1] = 0u;
      a.tiles[4 * tile + 2] = n_t;
      if (n_t) { s_tl_tile[ntl] = (uint32_t)tile; s_tl_pos[ntl] = nbuf; }
    }
    if (n_t) {
      // the values go through LDS so that only the set bits are visited
#pragma unroll
      for (int q = 0; q < G_VPT / 4; ++q) {
        u32x4 w;
#pragma unroll
        for (int i = 0; i < 4; ++i) w[i] = __float_as_uint(v[4 * q + i]);
        *reinterpret_cast<u32x4*>(&s_vals[threadIdx.x * G_VPT + 4 * q]) = w;
      }
      off += nbuf;
      for (uint32_t m = bm; m; m &= m - 1u) {
        const uint32_t bits = s_vals[threadIdx.x * G_VPT + (uint32_t)__builtin_ctz(m)];
        s_cand[off++] = bits;
        if (count_digits) atomicAdd(&s_bd[((bits & 0x7FFFFFFFu) >> 19) - blo], 1u);
      }
      nbuf += n_t;
      ++ntl;
    }
  }
  if (nbuf) flush();
  block_minmax<G_NT>(amin, amax, s_mm);
  const uint32_t cs = blockIdx.x % NSLOT;
  if (count_digits && threadIdx.x <= bhi - blo && s_bd[threadIdx.x])
    add_agent(&st[SP_BD + cs * BD_MAX + threadIdx.x], s_bd[threadIdx.x]);
  if (threadIdx.x == 0) {
    if (above_all) add_agent(slot(st, SP_ABOVE, cs), above_all);
    if (amin <= amax) {
      __hip_atomic_fetch_max(slot(st, SP_AMIN, cs), ~order_key(amin), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_fetch_max(slot(st, SP_AMAX, cs), order_key(amax), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  if (!last_block(st)) return;
  // the decision, on the first wavefront: each lane loads its slots and
  // digit counts at once (one round trip), wavefront sums and a scan combine them
  if (threadIdx.x >= WAVE) return;
  const uint32_t lane = threadIdx.x;
  uint32_t abv = 0, ncv = 0, bad = 0, mnv = 0, mxv = 0;
  if (lane < NSLOT) {
    abv = ld_agent(slot(st, SP_ABOVE, lane));
    mnv = ld_agent(slot(st, SP_AMIN, lane));
    mxv = ld_agent(slot(st, SP_AMAX, lane));
  }
  if (lane < a.n_sub) {
    ncv = ld_agent(slot(st, SP_NCAND, lane));
    bad = ncv > capc ? 1u : 0u;
  }
  // lane j: band digit bhi - j (the band's digits from the top)
  const uint32_t nd = bhi - blo + 1u;
  uint32_t cnt = 0;
  if (count_digits && lane < nd) {
    uint32_t c8[NSLOT];
#pragma unroll
    for (uint32_t c = 0; c < NSLOT; ++c) c8[c] = ld_agent(&st[SP_BD + c * BD_MAX + (bhi - lane - blo)]);
#pragma unroll
    for (uint32_t c = 0; c < NSLOT; ++c) cnt += c8[c];
  }
  // counts are below 2^31 (seg_len < 2^31), so 32-bit sums do not wrap
  const uint32_t ab = wave_sum(abv), nc = wave_sum(ncv);
  const bool fits = wave_sum(bad) == 0u;
  const bool fast = fits && ab < a.k && a.k <= (uint64_t)ab + nc;
  uint32_t b1 = 0, need2 = 0;
  bool p1 = false;
  if (fast && count_digits) {
    const uint32_t need = (uint32_t)(a.k - ab);
    const uint32_t incl = wave_incl_scan(cnt);
    const uint64_t hit = __ballot(lane < nd && incl >= need);
    if (hit) {
      const uint32_t j = (uint32_t)__builtin_ctzll(hit);
      const uint32_t before = (uint32_t)__builtin_amdgcn_readlane((int)(incl - cnt), (int)j);
      b1 = bhi - j;
      need2 = need - before;
      p1 = true;
    }
  }
  // values above the band, for the kept list's min / max
  uint32_t amn = mnv, amx = mxv;
#pragma unroll
  for (int o = 1; o < NSLOT; o <<= 1) {
    amn = max(amn, (uint32_t)__shfl_xor((int)amn, o));
    amx = max(amx, (uint32_t)__shfl_xor((int)amx, o));
  }
  if (lane == 0) {
    st[ST_ABOVE] = ab;
    st[ST_FAST] = fast ? 1u : 0u;
    st[ST_NEED1] = fast ? (uint32_t)(a.k - ab) : (uint32_t)a.k;
    if (p1) {
      st[ST_B1] = b1;
      st[ST_NEED2] = need2;
      st[ST_P1] = 1u;
    }
    st[ST_AMIN] = amn;
    st[ST_AMAX] = amx;
  }
}

// f(value bits) over every candidate, on the first CAND_GRID workgroups
template <typename F>
__device__ __forceinline__ void for_candidates(const GlobalArgs& a, F&& f) {
  const uint32_t G = min(gridDim.x, CAND_GRID);
  if (blockIdx.x >= G) return;
  const uint64_t capc = sub_cap(a);
  for (uint32_t c = 0; c < a.n_sub; ++c) {
    const uint64_t n = min((uint64_t)a.state[SP_NCAND + SLOT_WORDS * c], capc);
    const uint32_t* list = a.cand + c * capc;
    // eight loads in flight per thread before any is used
    constexpr int U = 8;
    const uint64_t stride = (uint64_t)G * G_NT;
    for (uint64_t j0 = (uint64_t)blockIdx.x * G_NT + threadIdx.x; j0 < n; j0 += U * stride) {
      uint32_t v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint64_t j = j0 + (uint64_t)u * stride;
        v[u] = (j < n) ? list[j] : 0u;
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (j0 + (uint64_t)u * stride < n) f(v[u]);
    }
  }
}

// ------------------------------------------------------------- passes 1-3
template <typename InT, bool EF, int PASS>
__global__ __launch_bounds__(G_NT) void k_g_pass(GlobalArgs a) {
  constexpr int NB = (PASS == 3) ? LAST_BINS : HIST_BINS;
  __shared__ uint32_t hist[NB];
  __shared__ uint32_t scratch[G_NT / WAVE + 2];
  __shared__ uint32_t found[2];
  uint32_t* st = a.state;
  if (PASS == 1 && st[ST_P1] != 0u) return;   // the band pass found the first digit
  const bool fast = st[ST_FAST] != 0u;
  // the candidate list is read by the first CAND_GRID workgroups only; the
  // rest leave at once and do not count towards the last workgroup
  const uint32_t G = fast ? min(gridDim.x, CAND_GRID) : gridDim.x;
  if (blockIdx.x >= G) return;
  zero_lds_bins(hist, NB);
  __syncthreads();
  const uint32_t b1 = (PASS >= 2) ? st[ST_B1] : 0u;
  const uint32_t p24 = (PASS == 3) ? ((st[ST_B1] << 12) | st[ST_B2]) : 0u;
  uint32_t zc = 0;
  auto count = [&](uint32_t kk) {
    bool in;
    uint32_t d;
    if constexpr (PASS == 1) { in = true; d = kk >> 19; }
    else if constexpr (PASS == 2) { in = (kk >> 19) == b1; d = (kk >> 7) & 0xFFFu; }
    else { in = (kk >> 7) == p24; d = kk & 0x7Fu; }
    if (in) {
      if (kk == 0u) ++zc;
      else atomicAdd(&hist[d], 1u);
    }
  };
  if (fast) {
    for_candidates(a, [&](uint32_t bits) { count(bits & 0x7FFFFFFFu); });
  } else {
    for (uint64_t tile = blockIdx.x; tile < a.n_tiles; tile += gridDim.x) {
      const uint64_t t0 = tile * G_TILE + (uint64_t)threadIdx.x * G_VPT;
      const int nv = (int)min((uint64_t)G_VPT, sat_sub(a.L, t0));
      float v[G_VPT];
      load_tile_values<InT, EF>(a, t0, nv, v);
#pragma unroll
      for (int i = 0; i < G_VPT; ++i)
        if (i < nv) count(mag_key(v[i]));
    }
  }
  const uint32_t zs = wave_sum(zc);
  if (lane_id() == 0 && zs) atomicAdd(&hist[0], zs);
  __syncthreads();
  uint32_t* gh = a.hist + (uint64_t)PASS * HIST_BINS;   // histograms 1..3
  merge_bins(hist, gh, NB);
  if (!last_block(st, G)) return;
  take_bins(hist, gh, NB);
  const uint32_t need = (PASS == 1) ? st[ST_NEED1] : (PASS == 2) ? st[ST_NEED2] : st[ST_NEED3];
  find_bin<G_NT, NB>(hist, need, scratch, found);
  if (threadIdx.x == 0) {
    if constexpr (PASS == 1) { st[ST_B1] = found[0]; st[ST_NEED2] = need - found[1]; }
    else if constexpr (PASS == 2) { st[ST_B2] = found[0]; st[ST_NEED3] = need - found[1]; }
    else {
      st[ST_T] = (p24 << 7) | found[0];
      st[ST_R] = need - found[1];
    }
  }
}

// ------------------------------------------------------------------ keptmm
// Min / max of the kept values, from the candidate list (keys == T are the
// ties; keys > T in the list are kept) and the values above the band; tcount
// reads every candidate once and gathers these on the way.  The r kept ties
// are the lowest-indexed ones; the list does not keep indices, so when ties
// of both signs exist and only some are kept, the tie values can decide lo
// or hi only if no kept value lies beyond +-|T| on that side; then the
// quantization is left to qpack.
struct KeptMM {
  float mn = __builtin_inff(), mx = -__builtin_inff();
  uint32_t tp = 0, tn = 0;
  __device__ __forceinline__ void add(uint32_t bits, uint32_t T) {
    const uint32_t kk = bits & 0x7FFFFFFFu;
    if (kk > T) { const float v = __uint_as_float(bits); mn = fminf(mn, v); mx = fmaxf(mx, v); }
    else if (kk == T) { if (bits >> 31) ++tn; else ++tp; }
  }
};

// the workgroup's part into the state (all threads call)
__device__ __forceinline__ void keptmm_push(uint32_t* st, KeptMM& m, uint32_t* scratch, float* s_mm) {
  block_minmax<G_NT>(m.mn, m.mx, s_mm);
  const uint32_t tps = block_sum<G_NT>(m.tp, scratch);
  const uint32_t tns = block_sum<G_NT>(m.tn, scratch);
  if (threadIdx.x == 0) {
    // the band pass's slots (already reduced into ST_AMIN / ST_AMAX, whose
    // values they still hold): one slot per eighth of the workgroups
    if (m.mn <= m.mx) {
      const uint32_t cs = blockIdx.x % NSLOT;
      __hip_atomic_fetch_max(slot(st, SP_AMIN, cs), ~order_key(m.mn), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_fetch_max(slot(st, SP_AMAX, cs), order_key(m.mx), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (tps) add_agent(&st[ST_TPOS], tps);
    if (tns) add_agent(&st[ST_TNEG], tns);
  }
}

// lo / hi / scale of the kept list, once every workgroup has pushed (one thread)
__device__ __forceinline__ void keptmm_final(const GlobalArgs& a, uint32_t* st) {
  const uint32_t T = st[ST_T];
  const uint32_t wmin = max(ld_agent(&st[ST_AMIN]), slot_max(st, SP_AMIN));
  const uint32_t wmax = max(ld_agent(&st[ST_AMAX]), slot_max(st, SP_AMAX));
  float lo = wmax ? from_order_key(~wmin) : __builtin_inff();
  float hi = wmax ? from_order_key(wmax) : -__builtin_inff();
  const uint32_t r = st[ST_R];
  const uint32_t np = ld_agent(&st[ST_TPOS]), nn = ld_agent(&st[ST_TNEG]);
  const float tf = __uint_as_float(T);
  bool pos_in = false, neg_in = false, ok = true;
  if (r == 0u) {
  } else if (r >= np + nn || T == 0u) {
    // every tie kept, or the ties are zeros (whose sign lo / hi lose anyway)
    pos_in = np > 0;
    neg_in = nn > 0;
  } else if (np > 0 && nn > 0) {
    // which sign the kept ties have is unknown here: harmless only if kept
    // values lie beyond both +|T| and -|T|
    ok = hi >= tf && lo <= -tf;
  } else {
    pos_in = np > 0;
    neg_in = nn > 0;
  }
  if (!ok) return;   // ST_PRE stays 0: qpack quantizes
  if (pos_in) { lo = fminf(lo, tf); hi = fmaxf(hi, tf); }
  if (neg_in) { lo = fminf(lo, -tf); hi = fmaxf(hi, -tf); }
  lo = lo + 0.0f;
  hi = hi + 0.0f;
  const uint32_t LV = (1u << a.bits) - 1u;
  const float scale = (hi != lo) ? (hi - lo) / (float)LV : 0.0f;
  st[ST_LO] = __float_as_uint(lo);
  st[ST_HI] = __float_as_uint(hi);
  st[ST_SCALE] = __float_as_uint(scale);
  st[ST_PRE] = 1u;
  a.meta[0] = lo;
  a.meta[1] = scale;
}

// ------------------------------------------------------------------ tcount
// Keys > T and == T per tile (from the candidate list and the band's counts
// on the fast path, else from the data), their exclusive prefix over each
// workgroup's contiguous range of tiles, and -- in the last workgroup -- the
// exclusive prefix of the workgroup totals.  emit then knows every tile's
// payload offset without waiting on other tiles.
constexpr uint32_t TC_GRID = 1024;   // tcount workgroups at most
constexpr uint32_t TPW_MAX = 512;    // tiles per tcount workgroup (segments < 2^31)
static_assert((uint64_t)TC_GRID * TPW_MAX * G_TILE >= (1ull << 31), "tile ranges cover 2^31 elements");
static_assert(TPW_MAX == 2 * G_NT, "two tiles per thread in the workgroup scan");

template <typename InT, bool EF>
__global__ __launch_bounds__(G_NT) void k_g_tcount(GlobalArgs a) {
  __shared__ uint32_t s_gt[TPW_MAX], s_eq[TPW_MAX];
  __shared__ uint32_t scratch[G_NT / WAVE + 2];
  __shared__ float s_mm[2 * (G_NT / WAVE)];
  uint32_t* st = a.state;
  const bool fast = st[ST_FAST] != 0u;
  const uint32_t T = st[ST_T];
  // the quantized kept list's min / max come from the candidates read here
  const bool mm = fast && a.bits != 0 && a.bits != 32;
  KeptMM kmm;
  const uint64_t t_lo = (uint64_t)blockIdx.x * a.tpw;
  const uint32_t nt = (uint32_t)min((uint64_t)a.tpw, sat_sub(a.n_tiles, t_lo));
  if (fast) {
    // one wavefront per tile, GT tiles of a wavefront at a time: their
    // records, then the first 2 * WAVE candidates of each, are loaded
    // together (two round trips per GT tiles instead of two per tile)
    constexpr uint32_t NW = G_NT / WAVE, GT = 4;
    const uint32_t w = threadIdx.x / WAVE, lane = (uint32_t)lane_id();
    auto take = [&](uint32_t bits, uint32_t& gt, uint32_t& eq) {
      const uint32_t kk = bits & 0x7FFFFFFFu;
      gt += kk > T;
      eq += kk == T;
      if (mm) kmm.add(bits, T);
    };
    for (uint32_t i0 = w; i0 < nt; i0 += NW * GT) {
      uint32_t ab[GT], off[GT], n[GT], c0[GT], c1[GT];
#pragma unroll
      for (uint32_t r = 0; r < GT; ++r) {
        const uint32_t i = i0 + r * NW;
        ab[r] = off[r] = n[r] = 0u;
        if (i < nt) {
          const uint32_t* rec = a.tiles + 4 * (t_lo + i);
          ab[r] = rec[0];
          off[r] = rec[1];
          n[r] = rec[2];
        }
      }
#pragma unroll
      for (uint32_t r = 0; r < GT; ++r) {
        const bool ok = (uint64_t)off[r] + n[r] <= a.cand_cap;
        c0[r] = (ok && lane < n[r]) ? a.cand[off[r] + lane] : 0u;
        c1[r] = (ok && lane + WAVE < n[r]) ? a.cand[off[r] + lane + WAVE] : 0u;
      }
#pragma unroll
      for (uint32_t r = 0; r < GT; ++r) {
        const uint32_t i = i0 + r * NW;
        uint32_t gt = 0, eq = 0;
        if ((uint64_t)off[r] + n[r] <= a.cand_cap) {
          if (lane < n[r]) take(c0[r], gt, eq);
          if (lane + WAVE < n[r]) take(c1[r], gt, eq);
          for (uint32_t j = lane + 2 * WAVE; j < n[r]; j += WAVE) take(a.cand[off[r] + j], gt, eq);
        } else if (lane == 0) {
          raise_error(KERR_INTERNAL);
        }
        gt = wave_sum(gt);
        eq = wave_sum(eq);
        if (lane == 0 && i < nt) { s_gt[i] = ab[r] + gt; s_eq[i] = eq; }
      }
    }
  } else {
    for (uint32_t i = 0; i < nt; ++i) {
      const uint64_t t0 = (t_lo + i) * G_TILE + (uint64_t)threadIdx.x * G_VPT;
      const int nv = (int)min((uint64_t)G_VPT, sat_sub(a.L, t0));
      float v[G_VPT];
      load_tile_values<InT, EF>(a, t0, nv, v);
      uint32_t gt = 0, eq = 0;
#pragma unroll
      for (int q = 0; q < G_VPT; ++q) {
        if (q < nv) {
          const uint32_t kk = mag_key(v[q]);
          gt += kk > T;
          eq += kk == T;
        }
      }
      const uint32_t tot = block_sum<G_NT>(gt | (eq << 16), scratch);
      if (threadIdx.x == 0) { s_gt[i] = tot & 0xFFFFu; s_eq[i] = tot >> 16; }
    }
  }
  __syncthreads();
  // exclusive prefix over the workgroup's tiles, two per thread
  const uint32_t i0 = 2 * threadIdx.x, i1 = i0 + 1;
  const uint32_t g0 = (i0 < nt) ? s_gt[i0] : 0u, g1 = (i1 < nt) ? s_gt[i1] : 0u;
  const uint32_t e0 = (i0 < nt) ? s_eq[i0] : 0u, e1 = (i1 < nt) ? s_eq[i1] : 0u;
  uint32_t gtot, etot;
  const uint32_t gx = block_excl_scan<G_NT>(g0 + g1, scratch, gtot);
  const uint32_t ex = block_excl_scan<G_NT>(e0 + e1, scratch, etot);
  if (i0 < nt) {
    uint32_t* rec = a.tiles + 4 * (t_lo + i0);
    rec[0] = g0; rec[1] = e0; rec[2] = gx; rec[3] = ex;
  }
  if (i1 < nt) {
    uint32_t* rec = a.tiles + 4 * (t_lo + i1);
    rec[0] = g1; rec[1] = e1; rec[2] = gx + g0; rec[3] = ex + e0;
  }
  if (threadIdx.x == 0) {
    st_agent(&a.wgs[2 * blockIdx.x], gtot);
    st_agent(&a.wgs[2 * blockIdx.x + 1], etot);
  }
  if (mm) keptmm_push(st, kmm, scratch, s_mm);
  if (!last_block(st)) return;
  if (mm && threadIdx.x == 0) keptmm_final(a, st);
  // exclusive prefix of the workgroup totals, four per thread
  constexpr int PER = (int)(TC_GRID / G_NT);
  uint32_t gw[PER], ew[PER], gs = 0, es = 0;
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const uint32_t wi = threadIdx.x * PER + q;
    gw[q] = (wi < gridDim.x) ? ld_agent(&a.wgs[2 * wi]) : 0u;
    ew[q] = (wi < gridDim.x) ? ld_agent(&a.wgs[2 * wi + 1]) : 0u;
    gs += gw[q];
    es += ew[q];
  }
  uint32_t dummy;
  uint32_t gp = block_excl_scan<G_NT>(gs, scratch, dummy);
  uint32_t ep = block_excl_scan<G_NT>(es, scratch, dummy);
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const uint32_t wi = threadIdx.x * PER + q;
    if (wi < gridDim.x) {
      a.wgs[2 * wi] = gp;
      a.wgs[2 * wi + 1] = ep;
    }
    gp += gw[q];
    ep += ew[q];
  }
}

// ------------------------------------------------------------------- emit
template <uint32_t B>
__device__ __forceinline__ uint32_t quant_code(float x, float lo, float range) {
  constexpr uint32_t LV = (1u << B) - 1u;
  if (!(range > 0.0f)) return 0u;
  const float u = (x - lo) / range;
  const float t = u * (float)LV;
  return min((uint32_t)rintf(t), LV);
}

// codes of entries [f, f + n) of the payload (c[j - f], B bits each), into
// the words they cover; a word not wholly inside the range is OR-ed in (the
// words start at zero), the rest are stored
template <uint32_t B, typename CT>
__device__ __forceinline__ void write_codes(uint32_t* codes, uint64_t wpg, uint64_t f, uint32_t n, const CT* c,
                                            bool shared_edges) {
  if (n == 0) return;
  const uint64_t b0 = f * B, b1 = (f + n) * B;   // bit range
  const uint64_t w0 = b0 / 32, w1 = (b1 - 1) / 32;
  for (uint64_t w = w0 + threadIdx.x; w <= w1; w += G_NT) {
    const uint64_t wb = w * 32;
    const uint64_t j0 = max(wb / B, f), j1 = min((wb + 31) / B, f + n - 1);
    uint32_t word = 0;
    for (uint64_t j = j0; j <= j1; ++j) {
      const int64_t o = (int64_t)(j * B) - (int64_t)wb;
      const uint32_t code = (uint32_t)c[j - f];
      word |= (o >= 0) ? (code << (uint32_t)o) : (code >> (uint32_t)(-o));
    }
    if (w >= wpg) { raise_error(KERR_INTERNAL); continue; }
    const bool inside = wb >= b0 && wb + 32 <= b1;
    if (inside || !shared_edges) codes[w] = word;
    else if (word) __hip_atomic_fetch_or(&codes[w], word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Q = 0: TopK values in the input dtype; Q = b: the kept list quantized.
// Per tile: (1) every thread marks its kept entries (bit masks), the tile's
// values go to LDS and the kept entries' offsets are compacted there; (2)
// the kept entries alone (about one in ten) are encoded, written to the
// payload, and their residual replaces the value in LDS; (3) the dense
// residual leaves from LDS.  Per-element work is thus only the two key
// comparisons; the encoding runs on the compacted list.
template <typename InT, bool EF, uint32_t Q>
__global__ __launch_bounds__(G_NT) void k_g_emit(GlobalArgs a) {
  using R = typename Elem<InT>::raw;
  constexpr bool QK = Q != 0;
  constexpr bool CODES = QK && Q != 32;   // b-bit codes, packed from LDS
  __shared__ __attribute__((aligned(16))) uint32_t s_v[G_TILE];   // the tile's values (binary32 bits)
  __shared__ uint16_t s_off[G_TILE];        // kept entries' offsets in the tile, in order
  __shared__ uint8_t s_code[CODES ? G_TILE : 1];
  __shared__ uint32_t scratch[G_NT / WAVE + 2];
  __shared__ float s_mm[2 * (G_NT / WAVE)];
  uint32_t* st = a.state;
  const bool none = a.k == 0;
  const uint32_t T = none ? 0u : st[ST_T];
  const uint32_t r = none ? 0u : st[ST_R];
  // quantize here when lo / hi are known (always for b = 32)
  const bool pre = QK && (Q == 32 || st[ST_PRE] != 0u);
  float lo = 0.0f, range = 0.0f, scale = 0.0f;
  if (CODES && pre) {
    lo = __uint_as_float(st[ST_LO]);
    range = __uint_as_float(st[ST_HI]) - lo;
    scale = __uint_as_float(st[ST_SCALE]);
  }
  float kmin = __builtin_inff(), kmax = -__builtin_inff();
  // Tiles from the last to the first: the band pass read them first to
  // last, so the last 256 MB it read are still in the on-package cache when
  // this pass starts (and the next micro-batch's band pass, which reads the
  // residual written here, starts where this pass ends).  Each tile's
  // payload offset comes from tcount, so the order is free.
  auto rev = [&](uint64_t i) { return a.n_tiles - 1 - i; };
  const bool pf = tiles_prefetchable(a);
  TileRaw<InT, EF> nxt;
  bool have = pf && tile_whole(a, rev(blockIdx.x));
  if (have) tile_fetch<InT, EF>(a, rev(blockIdx.x), nxt);
  for (uint64_t it = blockIdx.x; it < a.n_tiles; it += gridDim.x) {
    const uint64_t tile = rev(it);
    // the tile's offset (from tcount), loaded together with its data
    uint32_t gt_before = 0, eq_before = 0, rec_gt = 0, rec_eq = 0;
    if (!none) {
      // 8-byte loads: the workspace is 8-byte aligned
      const u32x2 cnt2 = *reinterpret_cast<const u32x2*>(a.tiles + 4 * tile);
      const u32x2 pre2 = *reinterpret_cast<const u32x2*>(a.tiles + 4 * tile + 2);
      const u32x2 wg2 = *reinterpret_cast<const u32x2*>(a.wgs + 2 * (tile / a.tpw));
      rec_gt = cnt2.x;
      rec_eq = cnt2.y;
      gt_before = wg2.x + pre2.x;
      eq_before = wg2.y + pre2.y;
    }
    const uint64_t t0 = tile * G_TILE + (uint64_t)threadIdx.x * G_VPT;
    const int nv = (int)min((uint64_t)G_VPT, sat_sub(a.L, t0));
    float v[G_VPT];
    if (have) tile_values<InT, EF>(nxt, v);
    else load_tile_values<InT, EF>(a, t0, nv, v);
    have = pf && it + gridDim.x < a.n_tiles && tile_whole(a, rev(it + gridDim.x));
    if (have) tile_fetch<InT, EF>(a, rev(it + gridDim.x), nxt);
    // ---- (1) keys > T and == T as bit masks (bit i: element i); keys
    // and T stay below 2^31, so the sign bit of a difference compares them
    uint32_t gm = 0, em = 0;
#pragma unroll
    for (int i = 0; i < G_VPT; ++i) {
      const uint32_t kk = mag_key(v[i]);
      gm |= ((T - kk) >> 31) << i;
      em |= (((kk ^ T) - 1u) >> 31) << i;
    }
    const uint32_t valid = (nv >= G_VPT) ? 0xFFFFu : ((1u << max(nv, 0)) - 1u);
    gm &= none ? 0u : valid;
    em &= none ? 0u : valid;
#pragma unroll
    for (int q = 0; q < G_VPT / 4; ++q) {
      u32x4 w;
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = __float_as_uint(v[4 * q + i]);
      *reinterpret_cast<u32x4*>(&s_v[threadIdx.x * G_VPT + 4 * q]) = w;
    }
    uint32_t tot;
    const uint32_t ex = block_excl_scan<G_NT>((uint32_t)__builtin_popcount(gm) | ((uint32_t)__builtin_popcount(em) << 16),
                                             scratch, tot);
    const uint32_t gt_t = tot & 0xFFFFu, eq_t = tot >> 16;
    if (!none && threadIdx.x == 0 && (rec_gt != gt_t || rec_eq != eq_t)) raise_error(KERR_INTERNAL);
    // ---- placement inside the tile (ties: the lowest indices overall)
    const uint32_t quota_t = min(sat_sub(r, eq_before), eq_t);
    const uint32_t gt_ex = ex & 0xFFFFu, eq_ex = ex >> 16;
    const uint32_t tile_first = gt_before + min(eq_before, r);
    const uint32_t cnt = gt_t + quota_t;
    uint32_t tie_keep = min(sat_sub(quota_t, eq_ex), (uint32_t)G_VPT);
    uint32_t km = gm, rest = em;             // kept: larger keys and the first tie_keep ties
    for (; tie_keep && rest; --tie_keep) {
      km |= rest & (0u - rest);
      rest &= rest - 1u;
    }
    uint32_t lp = gt_ex + min(eq_ex, quota_t);   // position in the tile's part of the payload
    if (lp + (uint32_t)__builtin_popcount(km) > G_TILE) {
      raise_error(KERR_INTERNAL);
      km = 0;
    }
    for (uint32_t m = km; m; m &= m - 1u) s_off[lp++] = (uint16_t)(threadIdx.x * G_VPT + (uint32_t)__builtin_ctz(m));
    if (a.blk && threadIdx.x == 0) a.blk[tile] = tile_first;
    __syncthreads();
    // ---- (2) the tile's kept entries, compacted: payload, and the
    // residual at their places in LDS
    const uint32_t n_ok = (uint32_t)min((uint64_t)cnt, sat_sub(a.k, (uint64_t)tile_first));
    if (n_ok < cnt && threadIdx.x == 0) raise_error(KERR_INTERNAL);
    for (uint32_t j = threadIdx.x; j < n_ok; j += G_NT) {
      const uint32_t off = s_off[j];
      const float x = __uint_as_float(s_v[off]);
      const uint64_t g = (uint64_t)tile_first + j;
      a.idx[g] = (uint32_t)(tile * G_TILE + off);
      float rec = x;   // what the receiver holds here (binary32 before its rounding)
      bool enc = true;
      if constexpr (!QK) ((R*)a.val)[g] = Elem<InT>::down(x);
      if constexpr (Q == 32) a.codes[g] = __float_as_uint(x);
      if constexpr (CODES) {
        if (pre) {
          const uint32_t c = quant_code<Q>(x, lo, range);
          s_code[j] = (uint8_t)c;
          const float prod = (float)c * scale;
          rec = lo + prod;
        } else {
          // without lo / hi the kept entries keep X in the residual and
          // qpack corrects them
          kmin = fminf(kmin, x);
          kmax = fmaxf(kmax, x);
          enc = false;
        }
      }
      if constexpr (EF) {
        if (enc) s_v[off] = __float_as_uint(x - through<InT>(rec));
      }
    }
    __syncthreads();
    if constexpr (CODES) {
      if (pre) write_codes<Q>(a.codes, a.wpg, tile_first, n_ok, s_code, true);
    }
    // ---- (3) the dense residual; write-back stores: the four 16-byte
    // stores of a thread fill each 128-byte line only together, which the
    // L2 merges before writing it
    if constexpr (EF) {
      float res[G_VPT];
#pragma unroll
      for (int q = 0; q < G_VPT / 4; ++q) {
        const u32x4 w = *reinterpret_cast<const u32x4*>(&s_v[threadIdx.x * G_VPT + 4 * q]);
#pragma unroll
        for (int i = 0; i < 4; ++i) res[4 * q + i] = __uint_as_float(w[i]);
      }
      if (nv > 0) store_run_partial<float, G_VPT, false>(a.e + t0, nv, res);
    }
    __syncthreads();
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    if (a.blk) a.blk[a.n_tiles] = (uint32_t)a.k;
    if constexpr (Q == 32) { a.meta[0] = 0.0f; a.meta[1] = 0.0f; }
  }
  if constexpr (CODES) {
    if (!pre) {
      block_minmax<G_NT>(kmin, kmax, s_mm);
      if (threadIdx.x == 0) push_minmax(st, ST_MIN, ST_MAX, kmin, kmax);
    }
  }
}

// ------------------------------------------------------------ qpack, clean
// Chunks of 8192 entries start on word boundaries for every b.
constexpr int QP_VPT = 32;
constexpr uint32_t QP_CH = (uint32_t)G_NT * QP_VPT;

// Only when emit could not quantize: codes of the kept list (one min-max
// group), meta, and the residual at the kept entries, where emit left X.
template <uint32_t B, typename OutT>
__device__ __forceinline__ void qpack_body(const GlobalArgs& a, uint8_t* s_code) {
  static_assert((QP_CH * B) % 32 == 0, "chunks on word boundaries");
  const uint32_t* st = a.state;
  constexpr uint32_t LV = (1u << B) - 1u;
  float lo = 0.0f, hi = 0.0f, scale = 0.0f;
  if (a.k > 0) {
    lo = from_order_key(~st[ST_MIN]) + 0.0f;
    hi = from_order_key(st[ST_MAX]) + 0.0f;
  }
  if (hi != lo) scale = (hi - lo) / (float)LV;
  const float range = hi - lo;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    a.meta[0] = lo;
    a.meta[1] = scale;
  }
  for (uint64_t c0 = (uint64_t)blockIdx.x * QP_CH; c0 < a.k; c0 += (uint64_t)gridDim.x * QP_CH) {
    const uint32_t n = (uint32_t)min((uint64_t)QP_CH, a.k - c0);
#pragma unroll 4
    for (int i = 0; i < QP_VPT; ++i) {
      const uint32_t jl = (uint32_t)i * G_NT + threadIdx.x;
      if (jl < n) {
        const uint32_t ix = a.idx[c0 + jl];
        uint32_t c = 0;
        if (ix < a.L) {
          const float x = a.e[ix];
          c = quant_code<B>(x, lo, range);
          const float prod = (float)c * scale;
          const float rec = lo + prod;
          a.e[ix] = x - through<OutT>(rec);
        } else {
          raise_error(KERR_INTERNAL);
        }
        s_code[jl] = (uint8_t)c;
      }
    }
    __syncthreads();
    write_codes<B>(a.codes, a.wpg, c0, n, s_code, false);
    __syncthreads();
  }
}

// The chain's last kernel.  B != 0 (the quantized kept list): first the
// qpack work when emit could not quantize.  Then back to the zero-filled
// workspace: tile words, the used part of the candidate list (its offset
// depends on the segment length, so a later call may find tile words there),
// then the state words (the last workgroup, once every workgroup has read
// the candidate counts and the state).
template <uint32_t B, typename OutT>
__global__ __launch_bounds__(G_NT) void k_g_finish(GlobalArgs a) {
  __shared__ uint8_t s_code[B ? QP_CH : 1];
  uint32_t* st = a.state;
  if constexpr (B != 0) {
    if (st[ST_PRE] == 0u) qpack_body<B, OutT>(a, s_code);   // k == 0 too: meta (0, 0)
  }
  const uint64_t gsz = (uint64_t)gridDim.x * G_NT, t = (uint64_t)blockIdx.x * G_NT + threadIdx.x;
  for (uint64_t i = t; i < 4 * a.n_tiles; i += gsz) st_agent(&a.tiles[i], 0u);
  for (uint64_t i = t; i < 2 * TC_GRID; i += gsz) st_agent(&a.wgs[i], 0u);
  const uint64_t capc = sub_cap(a);
  for (uint32_t c = 0; c < a.n_sub; ++c) {
    const uint64_t n = min((uint64_t)st[SP_NCAND + SLOT_WORDS * c], capc);
    for (uint64_t i = t; i < n; i += gsz) st_agent(&a.cand[c * capc + i], 0u);
  }
  if (!last_block(st)) return;
  for (int i = threadIdx.x; i < ST_WORDS; i += G_NT) st_agent(&st[i], 0u);
}

// ------------------------------------------------------------------ plans
namespace {

template <typename InT, bool EF>
const void* chain_ptr(int which) {
  switch (which) {
    case 0: return (const void*)k_g_sample<InT, EF>;
    case 1: return (const void*)k_g_band<InT, EF>;
    case 2: return (const void*)k_g_pass<InT, EF, 1>;
    case 3: return (const void*)k_g_pass<InT, EF, 2>;
    case 4: return (const void*)k_g_pass<InT, EF, 3>;
    case 5: return (const void*)k_g_tcount<InT, EF>;
  }
  return nullptr;
}
const void* pick_chain(int dt, bool ef, int which) {
  if (dt == DT_F32) return ef ? chain_ptr<float, true>(which) : chain_ptr<float, false>(which);
  if (dt == DT_BF16) return ef ? chain_ptr<bf16_t, true>(which) : chain_ptr<bf16_t, false>(which);
  return ef ? chain_ptr<f16_t, true>(which) : chain_ptr<f16_t, false>(which);
}

template <typename InT>
const void* emit_ptr(bool ef, uint32_t q) {
  if (q == 0) return ef ? (const void*)k_g_emit<InT, true, 0> : (const void*)k_g_emit<InT, false, 0>;
  if (!ef) return nullptr;
  switch (q) {
    case 1: return (const void*)k_g_emit<InT, true, 1>;
    case 2: return (const void*)k_g_emit<InT, true, 2>;
    case 3: return (const void*)k_g_emit<InT, true, 3>;
    case 4: return (const void*)k_g_emit<InT, true, 4>;
    case 5: return (const void*)k_g_emit<InT, true, 5>;
    case 6: return (const void*)k_g_emit<InT, true, 6>;
    case 7: return (const void*)k_g_emit<InT, true, 7>;
    case 8: return (const void*)k_g_emit<InT, true, 8>;
    case 32: return (const void*)k_g_emit<InT, true, 32>;
  }
  return nullptr;
}
const void* pick_emit(int dt, bool ef, uint32_t q) {
  if (dt == DT_F32) return emit_ptr<float>(ef, q);
  if (dt == DT_BF16) return emit_ptr<bf16_t>(ef, q);
  return emit_ptr<f16_t>(ef, q);
}

// the last kernel: qpack's work for b-bit kept lists (b = 0: none), then clean
template <typename OutT>
const void* finish_ptr(uint32_t b) {
  switch (b) {
    case 1: return (const void*)k_g_finish<1, OutT>;
    case 2: return (const void*)k_g_finish<2, OutT>;
    case 3: return (const void*)k_g_finish<3, OutT>;
    case 4: return (const void*)k_g_finish<4, OutT>;
    case 5: return (const void*)k_g_finish<5, OutT>;
    case 6: return (const void*)k_g_finish<6, OutT>;
    case 7: return (const void*)k_g_finish<7, OutT>;
    case 8: return (const void*)k_g_finish<8, OutT>;
  }
  return (const void*)k_g_finish<0, OutT>;
}
const void* pick_finish(int out_dt, uint32_t b) {
  if (out_dt == DT_F32) return finish_ptr<float>(b);
  if (out_dt == DT_BF16) return finish_ptr<bf16_t>(b);
  return finish_ptr<f16_t>(b);
}

hipError_t launch(const void* fn, uint32_t grid, uint32_t nt, const GlobalArgs& args, hipStream_t st) {
  if (!fn) return hipErrorInvalidValue;
  GlobalArgs a = args;
  void* params[] = {&a};
  return hipLaunchKernel(fn, dim3(grid), dim3(nt), params, 0, st);
}

// a tile loop's grid: no more workgroups than the compute units hold at once
// (the rest would start only when the first ones have gone through all
// their tiles, and run the last stretch at a fraction of the occupancy)
uint32_t resident_grid(const void* fn, uint32_t grid) {
  int per_cu = 0;
  if (!fn || hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, G_NT, 0) != hipSuccess || per_cu < 1) return grid;
  return std::max<uint32_t>(1, std::min<uint32_t>(grid, (uint32_t)per_cu * (uint32_t)device_cus()));
}

uint64_t cand_capacity(uint64_t L) { return L / 4 + 4096; }

}  // namespace

uint64_t global_ws_words(uint64_t L) {
  // state, four histograms, a record per tile, tcount's workgroup totals,
  // the candidate sub-lists
  return (uint64_t)ST_WORDS + 4ull * HIST_BINS + 4ull * n_blocks(L) + 2ull * TC_GRID + cand_capacity(L);
}

static uint32_t chain_grid(uint64_t n_tiles) {
  // eight workgroups per compute unit, each over many tiles
  return (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(n_tiles, (uint64_t)device_cus() * 8));
}

void global_ws_carve(uint32_t* ws, uint64_t L, GlobalArgs& a) {
  a.state = ws;
  a.hist = ws + ST_WORDS;
  a.tiles = ws + ST_WORDS + 4 * HIST_BINS;
  a.n_tiles = n_blocks(L);
  a.wgs = a.tiles + 4 * a.n_tiles;
  a.cand = a.wgs + 2 * TC_GRID;
  a.cand_cap = cand_capacity(L);
  a.sample_stride = (uint32_t)((a.n_tiles + SAMPLE_TILES - 1) / SAMPLE_TILES);
  a.n_sub = std::min<uint32_t>(chain_grid(a.n_tiles), NSLOT);
  const uint64_t tc_grid = std::max<uint64_t>(1, std::min<uint64_t>(a.n_tiles, TC_GRID));
  a.tpw = (uint32_t)((a.n_tiles + tc_grid - 1) / tc_grid);
}

hipError_t launch_global(int dt, bool ef, uint32_t qbits, const GlobalArgs& args, hipStream_t st) {
  // the quantized kept list needs the residual buffer (qpack reads X there)
  if (qbits != 0 && !ef) return hipErrorInvalidValue;
  const uint32_t grid = chain_grid(args.n_tiles);
  GlobalArgs a = args;
  if (a.n_sub < 1 || a.n_sub > NSLOT || a.n_sub > grid || a.tpw < 1 || a.tpw > TPW_MAX ||
      (a.n_tiles + a.tpw - 1) / a.tpw > TC_GRID)
    return hipErrorInvalidValue;
  a.bits = qbits;
  hipError_t e = hipSuccess;
  if (a.k > 0) {
    const uint64_t n_s = (a.n_tiles + a.sample_stride - 1) / a.sample_stride;
    const uint32_t sgrid = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(n_s, SAMPLE_GRID));
    e = launch(pick_chain(dt, ef, 0), sgrid, G_NT, a, st);
    for (int which = 1; which <= 4 && e == hipSuccess; ++which) {
      // band reads the whole segment; the digit passes read the candidate
      // list (CAND_GRID workgroups) unless the band missed, and are launched
      // with two workgroups per compute unit at most
      const void* fn = pick_chain(dt, ef, which);
      uint32_t g = resident_grid(fn, grid);
      if (which >= 2) g = std::min<uint32_t>(g, std::max<uint32_t>(CAND_GRID, 2u * (uint32_t)device_cus()));
      e = launch(fn, g, G_NT, a, st);
    }
    if (e == hipSuccess) {
      const uint32_t tgrid = (uint32_t)((a.n_tiles + a.tpw - 1) / a.tpw);
      e = launch(pick_chain(dt, ef, 5), tgrid, G_NT, a, st);
    }
  }
  if (e == hipSuccess) {
    const void* fn = pick_emit(dt, ef, qbits);
    e = launch(fn, resident_grid(fn, grid), G_NT, a, st);
  }
  if (e == hipSuccess) {
    const uint32_t qb = (qbits != 32) ? qbits : 0u;
    e = launch(pick_finish(dt, qb), std::min<uint32_t>(grid, 1024), G_NT, a, st);
  }
  return e;
}

TC_DEFINE_ERROR_READER(errors_global)

}  // namespace tc
