// tc_group.hpp -- exact TopK threshold for a segment spread over P
// workgroups whose values stay in registers (the group engine).
//
// TopK (Sec. 2.3 of the paper) keeps the k entries of largest magnitude.  The
// magnitude is the 31-bit key of mag_key(); the k-th largest key T and the
// tie quota r = k - #(key > T) define the kept set: key > T, or key == T and
// the entry is among the r lowest-index ties.
//
// Layout: workgroup `part` of a group owns the chunk [part*CH, part*CH + CH)
// of its segment; thread t holds R runs of E consecutive elements, run j at
// offset (j*NT + t)*E of the chunk (striped, so that every load and store
// instruction of a wavefront covers 1 KiB of contiguous memory).
//
// Two cross-workgroup exchanges per segment in the common case:
//   A. every workgroup adds its 4096-bin histogram of key bits 30..19 into
//      the group's histogram.  It also guesses, from its own keys, the bin
//      that holds the k-th largest key and adds 16 finer counts (bits 18..15)
//      for that bin and its two neighbours.  After the barrier, one read of
//      the merged counts gives the bin b1 and, when every workgroup's guess
//      covered b1, the 16-bit prefix of T.
//   B. every workgroup publishes a record: its count of keys above that
//      prefix and the keys that share it (a few per workgroup, carried
//      inline).  After the barrier each workgroup reads all records in one
//      round trip and finds T, the tie quota and what precedes it by itself.
// Otherwise (a guess missed, or too many keys share the prefix) the group
// goes on with 8-bit digit passes, each merged through device memory, and a
// last pass that publishes per-workgroup counts: exact for any input.
#pragma once

#include "tc_select.hpp"

namespace tc {

constexpr int GRP_NT = 512;
constexpr uint32_t GRP_MAX_P = 1024;      // workgroups per segment the engine supports
constexpr uint32_t REC_W = 64;            // words per record: above, count, inline keys
constexpr uint32_t REC_KEYS = REC_W - 2;
constexpr uint32_t FINE_SLOTS = 256;      // fine counts kept for bins b1 mod 256
constexpr uint32_t DIG_BINS = 256;        // 8-bit digits of the fallback passes
constexpr uint32_t DIG_ROWS = DIG_BINS + 1;   // per-workgroup slot: bins + larger-prefix count
constexpr uint32_t REC_P_MAX = 64;        // records of at most this many workgroups are read at once

// candidate keys the LDS list holds (records of up to 64 workgroups)
__host__ __device__ constexpr uint32_t grp_local_cap(uint32_t CH) { return CH > 4096u ? CH : 4096u; }

// Device memory owned by one group (inside the caller's workspace; zero on
// entry and left zero on exit), as word offsets from the group's base:
//   ctl[64]               [0] barrier arrivals (monotone during a launch), [1] exits
//   hist1[2][4096]        first-digit histograms, by segment parity
//   fine[2][256][16]      bits 18..15 of the keys in guessed bins, by bin mod 256
//   cov[2][256]           guesses per bin mod 256: count + (bin >> 8) << 16
//   hist2[4][256]         8-bit digit counts: [par] exchange B (bits 14..7), [2 + p]
//                         fallback pass p
//   rec[P][64]            exchange B records
//   slots[257][pitch]     last digit per workgroup + larger-prefix counts (fallback)
namespace gm_off {
constexpr uint32_t CTL = 0, HIST1 = 64, FINE = HIST1 + 2 * HIST_BINS, COV = FINE + 2 * FINE_SLOTS * 16,
                   HIST2 = COV + 2 * FINE_SLOTS, REC = HIST2 + 4 * DIG_BINS;
static_assert(REC % 4 == 0, "records are 16-byte aligned");
}  // namespace gm_off

__host__ __device__ constexpr uint64_t grp_mem_words(uint32_t P) {
  return gm_off::REC + (uint64_t)P * REC_W + (uint64_t)DIG_ROWS * slot_pitch(P);
}

// the group's memory: one base pointer, pieces at fixed offsets
struct GrpMem {
  uint32_t* base;
  uint32_t P;
  __device__ __forceinline__ uint32_t* ctl() const { return base + gm_off::CTL; }
  __device__ __forceinline__ uint32_t* hist1(uint32_t par) const { return base + gm_off::HIST1 + par * HIST_BINS; }
  __device__ __forceinline__ uint32_t* fine(uint32_t par) const { return base + gm_off::FINE + par * FINE_SLOTS * 16; }
  __device__ __forceinline__ uint32_t* cov(uint32_t par) const { return base + gm_off::COV + par * FINE_SLOTS; }
  __device__ __forceinline__ uint32_t* hist2(uint32_t q) const { return base + gm_off::HIST2 + q * DIG_BINS; }
  __device__ __forceinline__ uint32_t* rec() const { return base + gm_off::REC; }
  __device__ __forceinline__ uint32_t* slots() const { return base + gm_off::REC + P * REC_W; }
};

__device__ __forceinline__ GrpMem grp_mem(uint32_t* ws, uint32_t group, uint32_t P) {
  GrpMem g;
  g.base = ws + (uint64_t)group * grp_mem_words(P);
  g.P = P;
  return g;
}

// Barrier among the P workgroups of a group: arrivals are counted in one
// word that only grows during a launch, so the n-th barrier waits for n*P
// arrivals and nobody has to reset anything in flight.  Each wave's device-
// scope stores and atomics complete before its workgroup arrives.  Arrival
// and wait are separate calls so that a workgroup can do work of its own in
// between.  The wait is bounded (co-residency violated): it then raises
// KERR_TIMEOUT and returns.
__device__ __forceinline__ void group_arrive(uint32_t* ctr) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void group_wait(uint32_t* ctr, uint32_t target) {
  if (threadIdx.x == 0) {
    uint32_t spins = 0;
    while (ld_agent(ctr) < target) {
      __builtin_amdgcn_s_sleep(0);
      ++spins;
      if ((spins & 1023u) == 0u &&
          (__hip_atomic_load(&g_kernel_errors, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & KERR_TIMEOUT))
        break;
      if (spins > BARRIER_SPIN_LIMIT) { raise_error(KERR_TIMEOUT); break; }
    }
  }
  __syncthreads();
}
__device__ __forceinline__ void group_sync(uint32_t* ctr, uint32_t target) {
  group_arrive(ctr);
  group_wait(ctr, target);
}

// Exclusive scans of R values per thread across the workgroup in one pass;
// tot[j] = workgroup total of value j.  scratch: R * NT/64 words.
template <int NT, int R>
__device__ __forceinline__ void block_excl_scan_multi(const uint32_t (&v)[R], uint32_t (&ex)[R],
                                                      uint32_t (&tot)[R], uint32_t* scratch) {
  constexpr int NW = NT / WAVE;
  const int w = (int)threadIdx.x / WAVE;
  uint32_t incl[R];
#pragma unroll
  for (int j = 0; j < R; ++j) incl[j] = wave_incl_scan(v[j]);
  if (lane_id() == WAVE - 1) {
#pragma unroll
    for (int j = 0; j < R; ++j) scratch[j * NW + w] = incl[j];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < R; ++j) {
    uint32_t pre = 0, t = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const uint32_t x = scratch[j * NW + i];
      pre += (i < w) ? x : 0u;
      t += x;
    }
    ex[j] = pre + incl[j] - v[j];
    tot[j] = t;
  }
  __syncthreads();
}

// LDS of the group engine's selection
template <uint32_t CLOC>
struct GrpSelShared {
  uint32_t hist[HIST_BINS + WAVE];   // histograms (the last WAVE words: per-lane dummies)
  uint32_t cand[CLOC];               // exchange B records of all workgroups
};

struct GrpSmall {
  uint32_t scratch[8 * (GRP_NT / WAVE)];
  uint32_t found[2];
  uint32_t red[DIG_BINS];            // one digit's counts, copies summed
  uint32_t fwin[3 * 16 + WAVE];      // this workgroup's fine counts of its window
  uint32_t fmrg[3 * 16 + 3];         // the group's merged fine counts and coverage of that window
  uint32_t hist7[LAST_BINS + WAVE];  // last 7 bits of T (plus per-lane dummies)
  uint32_t misc[16];
  // this workgroup's keys on the 16-bit prefix, in index order (exchange B):
  // key, chunk offset, staged payload position
  uint32_t ckey[WAVE], coff[WAVE], cpos[WAVE];
  uint32_t rem[WAVE];                // staged positions dropped after exchange B, less their rank
};

// What exchange A leaves: the known leading bits of T, and the keys still to
// place below them.  fine: the 16-bit prefix is known (every workgroup's guess
// covered the bin of the k-th key).
struct SelA {
  uint32_t prefix, pbits, need;
  bool fine;
};

// Per-workgroup state carried across the segments a group handles.
struct GrpState {
  uint32_t nbar = 0;       // barriers passed (equal in all workgroups of the group)
  uint32_t iter = 0;       // segments handled
  bool used_slots = false; // the fallback ran (its words must be cleared on exit)
};

// Histogram copies for digit counts: values that repeat (differences of
// 16-bit numbers often do) would make the lanes of one wave hit one LDS
// address; with a copy per lane group (lane mod CP), spaced by an odd stride
// so that one bin's copies sit in distinct banks, at most 64/CP lanes meet.
// Word HS-1 of each copy absorbs lanes with nothing to count.
constexpr int DIG_CP = 16, DIG_HS = 257;
static_assert(DIG_CP * DIG_HS <= HIST_BINS + WAVE, "histogram copies fit the selection histogram");

template <int NT>
__device__ __forceinline__ void dig_zero(uint32_t* hist) {
  for (int i = (int)threadIdx.x; i < DIG_CP * DIG_HS; i += NT) hist[i] = 0u;
}
__device__ __forceinline__ void dig_add(uint32_t* hist, bool m, uint32_t digit) {
  const uint32_t base = (uint32_t)(lane_id() & (DIG_CP - 1)) * DIG_HS;
  atomicAdd(&hist[base + (m ? digit : (uint32_t)(DIG_HS - 1))], 1u);
}
// copies summed into red[0..NB); call after a barrier that follows the adds
template <int NT, int NB>
__device__ __forceinline__ void dig_reduce(const uint32_t* hist, uint32_t* red) {
  const int t = (int)threadIdx.x;
  if (t < NB) {
    uint32_t s = 0;
#pragma unroll
    for (int c = 0; c < DIG_CP; ++c) s += hist[c * DIG_HS + t];
    red[t] = s;
  }
}

// After the second barrier of a segment every workgroup has read the
// exchange A words of its parity: each clears a slice of them (histogram,
// fine counts and coverage lie back to back).
__device__ __forceinline__ void grp_clear_a(const GrpMem& g, uint32_t par, uint32_t P, uint32_t part) {
  const uint32_t n1 = HIST_BINS, n2 = FINE_SLOTS * 16, n3 = FINE_SLOTS;
  uint32_t* h1 = g.hist1(par);
  uint32_t* f1 = g.fine(par);
  uint32_t* c1 = g.cov(par);
  for (uint32_t i = part * GRP_NT + threadIdx.x; i < n1 + n2 + n3; i += P * GRP_NT) {
    uint32_t* p = (i < n1) ? h1 + i : (i < n1 + n2) ? f1 + (i - n1) : c1 + (i - n1 - n2);
    st_agent(p, 0u);
  }
}

// Exchange A for one segment held by the P workgroups of a group (this one
// is `part`), k >= 1.  v[j][i] is element i of this thread's run j.
// Elements past the segment's end hold +0: they have the smallest key and
// the highest indices, so with k <= L they rank after every real element and
// are never kept; the counts below need no bounds checks.  L: the segment's
// length, rounded to what the group covers when the guess scales k.
// Exchange A's first histogram (bits 30..19 of every key) and its window
// counts, cleared before the workgroup's values arrive, so that the keys of
// each run can be counted as soon as that run's loads land.
template <int NT, typename SH>
__device__ __forceinline__ void grp_hist_clear(SH& sh, GrpSmall& sm) {
  zero_lds<NT>(sh.hist, HIST_BINS);
  if (threadIdx.x < 3 * 16) sm.fwin[threadIdx.x] = 0u;
  __syncthreads();
}
// One key into it; exact zeros (common after a ReLU, and the padding) are
// counted in the thread's zc and added once per wave by exchange A, off one
// hot bin.
template <typename SH>
__device__ __forceinline__ void grp_hist_add(SH& sh, uint32_t kk, uint32_t& zc) {
  const uint32_t z = eq31(kk, 0u);
  zc += z;
  atomicAdd(&sh.hist[pick(z, HIST_BINS + (uint32_t)lane_id(), kk >> 19)], 1u);
}

// Exchange A proper: every key of the workgroup is in the first histogram
// (grp_hist_clear, then grp_hist_add per key; zc: this thread's exact zeros).
template <int NT, int R, int E, uint32_t CH>
__device__ __forceinline__ SelA grp_exchange_a(float (&v)[R][E], uint32_t zc, uint32_t k, uint64_t L, uint32_t P,
                                               uint32_t part, const GrpMem& g,
                                               GrpSelShared<grp_local_cap(CH)>& sh, GrpSmall& sm, GrpState& gs) {
  const int t = (int)threadIdx.x;
  auto key = [&](int j, int i) { return mag_key(v[j][i]); };
  const uint32_t par = gs.iter & 1u;

  // ---- A: the exact zeros into the first histogram, once per wave
  const uint32_t zs = wave_sum(zc);
  if (lane_id() == 0 && zs) atomicAdd(&sh.hist[0], zs);
  __syncthreads();

  uint32_t prefix, pbits, need;          // known leading bits of T, keys still to place
  bool fine = false;
  uint32_t lo = 0, hi = 0;
  if (P > 1) {
    // this workgroup's guess: its own bin at the same rank fraction
    const uint32_t need_loc = (uint32_t)min<uint64_t>(max<uint64_t>(((uint64_t)k * CH + L - 1) / L, 1), CH);
    find_bin<NT, HIST_BINS>(sh.hist, need_loc, sm.scratch, sm.found);
    const uint32_t bh = sm.found[0];
    lo = bh > 0u ? bh - 1u : 0u;
    hi = min(bh + 1u, (uint32_t)HIST_BINS - 1u);
    // bits 18..15 of the keys in bins lo..hi (the exact zeros, whose bits
    // 18..15 are 0, once per wave)
    refresh(v);
#pragma unroll
    for (int j = 0; j < R; ++j)
#pragma unroll
      for (int i = 0; i < E; ++i) {
        const uint32_t kk = key(j, i), b = kk >> 19;
        // in the window lo..hi (b - lo < 3, unsigned) and not an exact zero
        const uint32_t in = gt31(3u, b - lo) & (eq31(kk, 0u) ^ 1u) & (gt31(lo, b) ^ 1u);
        atomicAdd(&sm.fwin[pick(in, (b - lo) * 16u + ((kk >> 15) & 15u), 3u * 16u + (uint32_t)lane_id())], 1u);
      }
    if (lo == 0u && lane_id() == 0 && zs) atomicAdd(&sm.fwin[0], zs);
    __syncthreads();
    // merge into the group's counts
    uint32_t* h1 = g.hist1(par);
    uint32_t* f1 = g.fine(par);
    uint32_t* c1 = g.cov(par);
    for (int b = t; b < HIST_BINS; b += NT)
      if (sh.hist[b]) add_agent(&h1[b], sh.hist[b]);
    if (t < 3 * 16) {
      const uint32_t b = lo + (uint32_t)t / 16u;
      if (b <= hi && sm.fwin[t]) add_agent(&f1[(b & (FINE_SLOTS - 1)) * 16u + (uint32_t)t % 16u], sm.fwin[t]);
    } else if (t < 3 * 16 + 3) {
      const uint32_t b = lo + (uint32_t)(t - 3 * 16);
      if (b <= hi) add_agent(&c1[b & (FINE_SLOTS - 1)], 1u + ((b >> 8) << 16));
    }
    group_sync(g.ctl(), P * ++gs.nbar);
    // everybody has read the previous segment's exchange B counts: clear a slice
    if (gs.iter > 0)
      for (int b = (int)(part * NT) + t; b < (int)DIG_BINS; b += (int)(P * NT)) st_agent(&g.hist2(par ^ 1u)[b], 0u);
    // one round trip: the merged histogram, the fine counts and coverage of this window
    uint32_t fw = 0;
    if (t < 3 * 16 + 3) {
      const uint32_t b = lo + (uint32_t)(t < 48 ? t / 16 : t - 48);
      if (b <= hi) fw = ld_agent(t < 48 ? &f1[(b & (FINE_SLOTS - 1)) * 16u + (uint32_t)t % 16u] : &c1[b & (FINE_SLOTS - 1)]);
    }
    find_bin_global<NT>(h1, k, sm.scratch, sm.found);
    const uint32_t b1 = sm.found[0];
    need = k - sm.found[1];
    if (t < 3 * 16 + 3) sm.fmrg[t] = fw;
    __syncthreads();
    fine = b1 >= lo && b1 <= hi && sm.fmrg[48 + (b1 - lo)] == P + ((P * (b1 >> 8)) << 16);
    prefix = b1;
    pbits = 12;
    if (fine) {
      // bits 18..15 of T from the merged fine counts of b1 (every thread alike)
      const uint32_t* f = &sm.fmrg[(b1 - lo) * 16u];
      uint32_t acc = 0, f1v = 16;
      for (int q = 15; q >= 0; --q) {
        const uint32_t c = f[q];
        if (acc < need && need <= acc + c) { f1v = (uint32_t)q; break; }
        acc += c;
      }
      if (f1v < 16) {
        prefix = (b1 << 4) | f1v;
        pbits = 16;
        need -= acc;
      } else {
        fine = false;   // inconsistent counts: never expected; take the exact passes
      }
    }
    __syncthreads();
  } else {
    find_bin<NT, HIST_BINS>(sh.hist, k, sm.scratch, sm.found);
    prefix = sm.found[0];
    pbits = 12;
    need = k - sm.found[1];
    __syncthreads();
  }
  SelA A;
  A.prefix = prefix;
  A.pbits = pbits;
  A.need = need;
  A.fine = fine;
  return A;
}

// Exchange B (fine mode), first half.  Before calling, this workgroup has
// written the keys that share the 16-bit prefix into its record (slots 2..,
// at most REC_KEYS of them), counted their bits 14..7 into sm.red (followed
// by a barrier), and knows how many of its keys lie above the prefix
// (abv_wg) and on it (cnt_wg).  Publishes the counts and arrives at the
// group's barrier; the workgroup may work on its own until grp_finish_b.
template <int NT>
__device__ __forceinline__ void grp_publish_b(uint32_t part, const GrpMem& g, const GrpSmall& sm, GrpState& gs,
                                              uint32_t abv_wg, uint32_t cnt_wg) {
  const int t = (int)threadIdx.x;
  uint32_t* my = g.rec() + (uint64_t)part * REC_W;
  uint32_t* h2 = g.hist2(gs.iter & 1u);
  if (t < (int)DIG_BINS && sm.red[t]) add_agent(&h2[t], sm.red[t]);
  if (t == 0) { st_agent(&my[0], abv_wg); st_agent(&my[1], cnt_wg); }
  ++gs.nbar;
  group_arrive(g.ctl());
}

// Exchange B, second half: waits for the group, reads all records and the
// merged digit counts in one round trip and finds T, the tie quota and the
// larger keys and ties of lower workgroups (the last after one more barrier,
// by grp_finish_b_lower).  Returns false (nothing decided)
// when some record could not hold its keys; exchange A's words are cleared
// either way.
template <int NT>
__device__ __forceinline__ bool grp_finish_b(uint32_t k, uint32_t P, uint32_t part, const GrpMem& g, GrpSmall& sm,
                                             GrpState& gs, const SelA& A, SelResult& res) {
  constexpr int NW = NT / WAVE;
  constexpr int SPT = (int)(REC_P_MAX * REC_W / NT);
  static_assert(NT % REC_W == 0 && REC_W == WAVE, "a record is one word per lane of a wavefront");
  const int t = (int)threadIdx.x, wv = t / WAVE, lane = lane_id();
  const uint32_t par = gs.iter & 1u;
  group_wait(g.ctl(), P * gs.nbar);
  grp_clear_a(g, par, P, part);
  // lane i of wavefront wv reads word i of records u*NW + wv
  uint32_t hd = 0;
  if (t < (int)DIG_BINS) hd = ld_agent(&g.hist2(par)[t]);
  const uint32_t* rec = g.rec();
  uint32_t wd[SPT];
#pragma unroll
  for (int u = 0; u < SPT; ++u) {
    const uint32_t w = (uint32_t)(u * NW + wv);
    wd[u] = (w < P) ? ld_agent(&rec[(uint64_t)w * REC_W + (uint32_t)lane]) : 0u;
  }
  // totals from the record headers (words 0 and 1 sit in lanes 0 and 1)
  uint32_t cnt[SPT], abv_bef = 0, abv_all = 0, bad = 0;
#pragma unroll
  for (int u = 0; u < SPT; ++u) {
    const uint32_t w = (uint32_t)(u * NW + wv);
    const uint32_t aw = __builtin_amdgcn_readlane(wd[u], 0);
    cnt[u] = __builtin_amdgcn_readlane(wd[u], 1);
    abv_all += aw;
    abv_bef += (w < part) ? aw : 0u;
    bad |= (cnt[u] > REC_KEYS) ? 1u : 0u;
  }
  uint32_t* tsc = sm.scratch + 5 * NW;   // clear of the scans' words
  if (lane == 0) { tsc[wv] = abv_bef; tsc[NW + wv] = abv_all; tsc[2 * NW + wv] = bad; }
  if (t < (int)DIG_BINS) sm.red[t] = hd;
  if (t < (int)LAST_BINS) sm.hist7[t] = 0u;
  __syncthreads();
  abv_bef = 0;
  abv_all = 0;
  bad = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) { abv_bef += tsc[i]; abv_all += tsc[NW + i]; bad |= tsc[2 * NW + i]; }
  if (bad != 0) return false;
  // bits 14..7 of T from the merged digit counts; bits 6..0 from the inline
  // keys that share the 24-bit prefix
  uint32_t c[SPT];
  bool lower[SPT];
#pragma unroll
  for (int u = 0; u < SPT; ++u) {
    const uint32_t w = (uint32_t)(u * NW + wv);
    const bool valid = lane >= 2 && (uint32_t)(lane - 2) < cnt[u];   // cnt is 0 past the last record
    c[u] = valid ? wd[u] : ~0u;           // ~0u matches no prefix
    lower[u] = valid && w < part;
  }
  const uint32_t need_b = k - abv_all;
  find_bin_wave<256>(sm.red, need_b, sm.found);
  const uint32_t p24 = (A.prefix << 8) | sm.found[0];
  const uint32_t need_c = need_b - sm.found[1];
  const uint32_t dummy = LAST_BINS + (uint32_t)lane;
#pragma unroll
  for (int u = 0; u < SPT; ++u) atomicAdd(&sm.hist7[(c[u] >> 7) == p24 ? (c[u] & 0x7Fu) : dummy], 1u);
  __syncthreads();
  find_bin_wave<LAST_BINS>(sm.hist7, need_c, sm.found);
  res.T = (p24 << 7) | sm.found[0];
  res.r = need_c - sm.found[1];
  // larger keys and ties in lower workgroups' records (both below 2^16),
  // summed per wavefront into sm.scratch[0..NW): grp_finish_b_lower adds
  // them up after the caller's next barrier
  uint32_t ge = 0;
#pragma unroll
  for (int u = 0; u < SPT; ++u)
    ge += (lower[u] && c[u] > res.T) ? 1u : ((lower[u] && c[u] == res.T) ? 0x10000u : 0u);
  ge = wave_sum(ge);
  if (lane == 0) sm.scratch[wv] = ge;
  res.gt_before = abv_bef;
  res.eq_before = 0;
  return true;
}

template <int NT>
__device__ __forceinline__ void grp_finish_b_lower(const GrpSmall& sm, SelResult& res) {
  uint32_t sge = 0;
#pragma unroll
  for (int i = 0; i < NT / WAVE; ++i) sge += sm.scratch[i];
  res.gt_before += sge & 0xFFFFu;
  res.eq_before = sge >> 16;
}

// The exact passes from the prefix exchange A (or B) left: 8-bit digit
// passes merged through device memory, then a last digit of at most 8 bits
// counted per workgroup (slots), which also gives what precedes this
// workgroup.  `cleared`: exchange A's words have already been cleared.
template <int NT, int R, int E, uint32_t CH>
__device__ __forceinline__ SelResult grp_fallback(float (&v)[R][E], uint32_t P, uint32_t part, const GrpMem& g,
                                                  GrpSelShared<grp_local_cap(CH)>& sh, GrpSmall& sm, GrpState& gs,
                                                  uint32_t prefix, uint32_t pbits, uint32_t need, bool cleared) {
  const int t = (int)threadIdx.x;
  auto key = [&](int j, int i) { return mag_key(v[j][i]); };
  const uint32_t par = gs.iter & 1u;
  SelResult res;
  gs.used_slots = gs.used_slots || P > 1;
  for (int pass = 0; 31u - pbits > 8u; ++pass) {
    const uint32_t sh8 = 31u - pbits - 8u;         // the digit's lowest bit
    dig_zero<NT>(sh.hist);
    __syncthreads();
    refresh(v);
#pragma unroll
    for (int j = 0; j < R; ++j)
#pragma unroll
      for (int i = 0; i < E; ++i) {
        const uint32_t kk = key(j, i);
        dig_add(sh.hist, (kk >> (sh8 + 8u)) == prefix, (kk >> sh8) & 0xFFu);
      }
    __syncthreads();
    dig_reduce<NT, 256>(sh.hist, sm.red);
    __syncthreads();
    if (P > 1) {
      // at most two passes per segment, each with its own counts (cleared
      // after the last-digit barrier)
      uint32_t* h2 = g.hist2(2u + (uint32_t)pass);
      if (t < (int)DIG_BINS && sm.red[t]) add_agent(&h2[t], sm.red[t]);
      group_sync(g.ctl(), P * ++gs.nbar);
      if (t < (int)DIG_BINS) sm.red[t] = ld_agent(&h2[t]);
      if (!cleared) { grp_clear_a(g, par, P, part); cleared = true; }
      __syncthreads();
    }
    find_bin_wave<256>(sm.red, need, sm.found);
    prefix = (prefix << 8) | sm.found[0];
    pbits += 8;
    need -= sm.found[1];
    __syncthreads();
  }
  // last digit: per-workgroup counts, published as transposed slots
  const uint32_t lb = 31u - pbits;                  // 1..8 bits
  const uint32_t nbl = 1u << lb;
  dig_zero<NT>(sh.hist);
  __syncthreads();
  refresh(v);
  uint32_t gtp = 0;   // keys with a larger prefix
#pragma unroll
  for (int j = 0; j < R; ++j)
#pragma unroll
    for (int i = 0; i < E; ++i) {
      const uint32_t kk = key(j, i);
      dig_add(sh.hist, (kk >> lb) == prefix, kk & (nbl - 1u));
      gtp += ((kk >> lb) > prefix) ? 1u : 0u;
    }
  const uint32_t gtp_wg = block_sum<NT>(gtp, sm.scratch);   // contains barriers
  dig_reduce<NT, 256>(sh.hist, sm.red);
  __syncthreads();
  uint32_t* hall = sh.cand;                 // [256] whole segment
  uint32_t* hbef = sh.cand + DIG_BINS;      // [256] lower workgroups
  uint32_t gtpb = 0;
  if (P > 1) {
    const uint32_t pitch = slot_pitch(P);
    uint32_t* slots = g.slots();
    if (t < (int)DIG_BINS) st_agent(&slots[(uint64_t)t * pitch + part], sm.red[t]);
    if (t == 0) st_agent(&slots[(uint64_t)DIG_BINS * pitch + part], gtp_wg);
    group_sync(g.ctl(), P * ++gs.nbar);
    if (!cleared) { grp_clear_a(g, par, P, part); cleared = true; }
    // every digit pass has been read by everybody: clear a slice of their counts
    for (int b = (int)(part * NT) + t; b < (int)(2 * DIG_BINS); b += (int)(P * NT)) st_agent(&g.hist2(2)[b], 0u);
    // row `bin` of the slots holds that bin's count in every workgroup; two
    // thread sets split each row and read it in 8-byte pairs
    constexpr int SETS = NT / (int)DIG_BINS;
    const int bin = t % (int)DIG_BINS, set = t / (int)DIG_BINS;
    const uint32_t per = pitch / SETS;          // even: pitch is a multiple of 8
    const uint64_t* row = reinterpret_cast<const uint64_t*>(slots + (uint64_t)bin * pitch + set * per);
    uint32_t a_all = 0, a_bef = 0;
    for (uint32_t q = 0; q < per / 2; ++q) {
      const uint64_t pr = ld_agent64(row + q);
      const uint32_t jw = set * per + 2 * q;
      const uint32_t lo2 = (uint32_t)pr, hi2 = (uint32_t)(pr >> 32);
      a_all += lo2 + hi2;
      a_bef += (jw < part ? lo2 : 0u) + (jw + 1 < part ? hi2 : 0u);
    }
    uint32_t g_own = 0;
    for (uint32_t q = (uint32_t)t; q < part; q += NT) g_own += ld_agent(slots + (uint64_t)DIG_BINS * pitch + q);
    uint32_t* red = sh.hist;   // [SETS][2][256] partial sums (free now)
    red[(set * 2) * DIG_BINS + bin] = a_all;
    red[(set * 2 + 1) * DIG_BINS + bin] = a_bef;
    __syncthreads();
    if (t < (int)DIG_BINS) {
      uint32_t s_all = 0, s_bef = 0;
#pragma unroll
      for (int q = 0; q < SETS; ++q) { s_all += red[(q * 2) * DIG_BINS + t]; s_bef += red[(q * 2 + 1) * DIG_BINS + t]; }
      hall[t] = s_all;
      hbef[t] = s_bef;
    }
    gtpb = block_sum<NT>(g_own, sm.scratch);
  } else {
    if (t < (int)DIG_BINS) { hall[t] = sm.red[t]; hbef[t] = 0u; }
  }
  __syncthreads();
  find_bin_wave<256>(hall, need, sm.found);
  const uint32_t d = sm.found[0];
  res.T = (prefix << lb) | d;
  res.r = need - sm.found[1];
  const uint32_t gt_digit = (t < (int)DIG_BINS && (uint32_t)t > d) ? hbef[t] : 0u;
  res.gt_before = gtpb + block_sum<NT>(gt_digit, sm.scratch);
  res.eq_before = hbef[d];
  __syncthreads();
  return res;
}

// Leave the group's workspace zero.  Every workgroup takes an exit ticket
// once it has read the last exchange words (grp_exit_ticket: the atomic is
// issued, nobody waits for it); at its very end, the workgroup that drew the
// last ticket (all others have finished reading) clears the barrier words,
// the records, exchange B's digit counts of both parities and, if the
// fallback ran, the slots; everything else is cleared in flight.
__device__ __forceinline__ uint32_t grp_exit_ticket(const GrpMem& g) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  uint32_t prev = 0;
  if (threadIdx.x == 0) prev = __hip_atomic_fetch_add(g.ctl() + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return prev;   // thread 0's ticket; other threads' values are meaningless
}

template <int NT>
__device__ __forceinline__ void grp_exit_finish(const GrpMem& g, uint32_t P, const GrpState& gs, uint32_t ticket,
                                                uint32_t* flag) {
  if (threadIdx.x == 0) *flag = (ticket == P - 1) ? 1u : 0u;
  __syncthreads();
  if (!*flag) return;
  const uint64_t nrec = (uint64_t)P * REC_W;
  uint32_t* rec = g.rec();
  for (uint64_t i = threadIdx.x; i < nrec; i += NT) st_agent(&rec[i], 0u);
  for (uint32_t i = threadIdx.x; i < 2 * DIG_BINS; i += NT) st_agent(&g.hist2(0)[i], 0u);
  if (gs.used_slots) {
    const uint64_t n = (uint64_t)DIG_ROWS * slot_pitch(P);
    uint32_t* slots = g.slots();
    for (uint64_t i = threadIdx.x; i < n; i += NT) st_agent(&slots[i], 0u);
  }
  if (threadIdx.x == 0) {
    st_agent(g.ctl(), 0u);
    st_agent(g.ctl() + 1, 0u);
  }
}

}  // namespace tc
