// tc_select.hpp -- exact TopK threshold selection on register-resident keys.
//
// TopK (Sec. 2.3 of the paper) keeps the k entries of largest magnitude.  On
// the device the magnitude is the 31-bit key of mag_key(); the k-th largest
// key T and the tie quota r = k - #(key > T) define the kept set:
//   key > T, or key == T and the entry is among the r lowest-index ties.
//
// Two strategies, both exact:
//  * radix_select: three digit passes over the keys (bits 30..19, 18..7,
//    6..0) with LDS histograms.  A segment may be spread over P workgroups;
//    the first two passes merge their histograms with device-scope atomics,
//    the last pass publishes per-workgroup histograms ("slots") so that every
//    workgroup also learns how many larger keys and ties precede it.  Three
//    cross-workgroup barriers per segment.
//  * bitwise_select: one wavefront owns a whole short segment (a token row)
//    and fixes T bit by bit, counting with ballots; no LDS, no barriers.
#pragma once

#include "tc_device.hpp"

namespace tc {

constexpr int HIST_BINS = 4096;   // 12-bit digits for the first two passes
constexpr int LAST_BINS = 128;    // 7-bit digit for the last pass
constexpr int SLOT_ROWS = LAST_BINS + 1;   // per-workgroup slot: 128 bins + larger-prefix count
constexpr int CAND_CAP = 256;     // per-wave list of the keys inside the first-pass bin

// slot rows are laid out transposed, [row][workgroup], each row padded to a
// multiple of 8 workgroups so that readers can take them in 8-byte pairs
__host__ __device__ constexpr uint32_t slot_pitch(uint32_t P) { return (P + 7u) & ~7u; }

// device memory owned by one group of P workgroups (inside the caller's
// workspace, zero-filled before first use and left zero-filled on exit)
struct GroupMem {
  uint32_t* bar;     // [3] barrier count / sense / exit count
  uint32_t* hist1;   // [HIST_BINS]
  uint32_t* hist2;   // [HIST_BINS]
  uint32_t* slots;   // [SLOT_ROWS][slot_pitch(P)]
};

// words of workspace per group (barrier padded to 64 words)
__host__ __device__ constexpr uint64_t group_mem_words(uint32_t P) {
  return 64u + 2u * HIST_BINS + (uint64_t)SLOT_ROWS * slot_pitch(P);
}
__host__ __device__ constexpr uint64_t slot_words(uint32_t P) { return (uint64_t)SLOT_ROWS * slot_pitch(P); }

__device__ __forceinline__ GroupMem group_mem(uint32_t* ws, uint32_t group, uint32_t P) {
  uint32_t* base = ws + (uint64_t)group * group_mem_words(P);
  GroupMem g;
  g.bar = base;
  g.hist1 = base + 64;
  g.hist2 = base + 64 + HIST_BINS;
  g.slots = base + 64 + 2 * HIST_BINS;
  return g;
}

template <int NT>
struct SelShared {
  uint32_t hist[HIST_BINS];
  uint32_t cand[(NT / WAVE) * CAND_CAP];
  uint32_t scratch[NT / WAVE + 2];
  uint32_t found[2];          // bin, count above it
};

__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

struct SelResult {
  uint32_t T;          // threshold key (0xFFFFFFFF when k == 0: nothing kept)
  uint32_t r;          // ties at T to keep over the whole segment
  uint32_t gt_before;  // keys > T in lower-indexed workgroups of the segment
  uint32_t eq_before;  // keys == T in lower-indexed workgroups of the segment
};

// Find the bin b of a histogram with  sum_{c > b} h[c] < need <= sum_{c >= b} h[c]
// (1 <= need <= sum h), given each thread's BPT consecutive bins in loc[]
// (thread t owns bins [t*BPT, t*BPT + BPT)).  Writes (b, sum_{c > b} h[c])
// to found[].
template <int NT, int BPT>
__device__ __forceinline__ void find_bin_loc(const uint32_t (&loc)[BPT], uint32_t need, uint32_t* scratch,
                                             uint32_t* found) {
  const int t = (int)threadIdx.x;
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < BPT; ++i) sum += loc[i];
  uint32_t total;
  const uint32_t pre = block_excl_scan<NT>(sum, scratch, total);
  uint32_t acc = total - pre - sum;           // keys in bins owned by higher threads
  if (acc < need && need <= acc + sum) {
#pragma unroll
    for (int i = BPT - 1; i >= 0; --i) {
      if (acc + loc[i] >= need) { found[0] = (uint32_t)(t * BPT + i); found[1] = acc; break; }
      acc += loc[i];
    }
  }
  __syncthreads();
}

// ... with the histogram in LDS
template <int NT, int NB>
__device__ __forceinline__ void find_bin(const uint32_t* h, uint32_t need, uint32_t* scratch, uint32_t* found) {
  constexpr int BPT = (NB + NT - 1) / NT;
  uint32_t loc[BPT];
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int b = (int)threadIdx.x * BPT + i;
    loc[i] = (b < NB) ? h[b] : 0u;
  }
  find_bin_loc<NT, BPT>(loc, need, scratch, found);
}

// ... with the merged histogram in device memory (read with device-scope
// 8-byte loads straight into registers)
template <int NT>
__device__ __forceinline__ void find_bin_global(const uint32_t* gh, uint32_t need, uint32_t* scratch,
                                                uint32_t* found) {
  constexpr int BPT = HIST_BINS / NT;
  static_assert(BPT >= 2 && BPT % 2 == 0, "two bins per 8-byte load");
  uint32_t loc[BPT];
  const uint64_t* p = reinterpret_cast<const uint64_t*>(gh + threadIdx.x * BPT);
#pragma unroll
  for (int i = 0; i < BPT / 2; ++i) {
    const uint64_t w = ld_agent64(p + i);
    loc[2 * i] = (uint32_t)w;
    loc[2 * i + 1] = (uint32_t)(w >> 32);
  }
  find_bin_loc<NT, BPT>(loc, need, scratch, found);
}

// Count this workgroup's keys that match `prefix` under `pmask` into LDS bins
// by `digit = (key >> shift) & dmask`.  Zero keys (exact zeros are common in
// ReLU outputs) are counted in registers and added once per wave, which keeps
// them off a single hot LDS address.
template <int NT, int VPT>
__device__ __forceinline__ void count_digits(const uint32_t (&key)[VPT], int nv, uint32_t pshift,
                                             uint32_t prefix, uint32_t shift, uint32_t dmask,
                                             uint32_t* hist) {
  uint32_t zc = 0;
#pragma unroll
  for (int v = 0; v < VPT; ++v) {
    if (v < nv) {
      const uint32_t kk = key[v];
      if ((kk >> pshift) == prefix) {
        if (kk == 0u) ++zc;
        else atomicAdd(&hist[(kk >> shift) & dmask], 1u);
      }
    }
  }
  const uint32_t zs = wave_sum(zc);
  if (lane_id() == 0 && zs) atomicAdd(&hist[0], zs);
}

template <int NT>
__device__ __forceinline__ void zero_lds(uint32_t* h, int n) {
  for (int b = (int)threadIdx.x; b < n; b += NT) h[b] = 0u;
}

// Exact threshold for one segment spread over P workgroups (this one is
// `part`), with k >= 1 entries to keep out of the segment's valid keys.
template <int NT, int VPT>
__device__ SelResult radix_select(const uint32_t (&key)[VPT], int nv, uint32_t k, uint32_t P,
                                  uint32_t part, const GroupMem& g, SelShared<NT>& sh) {
  static_assert(NT >= 2 * LAST_BINS, "the slot gather splits the workgroup over the last-digit bins");
  SelResult res;
  const int t = (int)threadIdx.x;
  // ---- pass 1: bits 30..19 of all keys
  zero_lds<NT>(sh.hist, HIST_BINS);
  __syncthreads();
  count_digits<NT, VPT>(key, nv, 31, 0u, 19, 0xFFFu, sh.hist);
  __syncthreads();
  if (P > 1) {
    for (int b = t; b < HIST_BINS; b += NT)
      if (sh.hist[b]) add_agent(&g.hist1[b], sh.hist[b]);
    group_barrier(g.bar, P);
    find_bin_global<NT>(g.hist1, k, sh.scratch, sh.found);
  } else {
    find_bin<NT, HIST_BINS>(sh.hist, k, sh.scratch, sh.found);
  }
  const uint32_t b1 = sh.found[0];
  const uint32_t need2 = k - sh.found[1];
  __syncthreads();

  // ---- the keys inside bin b1 go to a per-wave list in LDS (ballot
  // compaction), so that the next two passes touch only them
  const int w = t / WAVE;
  uint32_t* cand = sh.cand + w * CAND_CAP;
  uint32_t ccount = 0;   // wave-uniform
  uint32_t gt1 = 0;      // keys above bin b1
#pragma unroll
  for (int v = 0; v < VPT; ++v) {
    const bool valid = v < nv;
    const uint32_t kk = key[v];
    const bool in = valid && (kk >> 19) == b1;
    gt1 += (valid && (kk >> 19) > b1) ? 1u : 0u;
    const uint64_t bal = __ballot(in);
    if (in) {
      const uint32_t slot = ccount + lanes_below(bal);
      if (slot < (uint32_t)CAND_CAP) cand[slot] = kk;
    }
    ccount += (uint32_t)__popcll(bal);
  }
  const bool listed = ccount <= (uint32_t)CAND_CAP;   // else this wave counts from registers

  // ---- pass 2: bits 18..7 of keys whose bits 30..19 equal b1
  zero_lds<NT>(sh.hist, HIST_BINS);
  __syncthreads();
  if (listed) {
    for (uint32_t i = (uint32_t)lane_id(); i < ccount; i += WAVE) atomicAdd(&sh.hist[(cand[i] >> 7) & 0xFFFu], 1u);
  } else {
    count_digits<NT, VPT>(key, nv, 19, b1, 7, 0xFFFu, sh.hist);
  }
  __syncthreads();
  if (P > 1) {
    for (int b = t; b < HIST_BINS; b += NT)
      if (sh.hist[b]) add_agent(&g.hist2[b], sh.hist[b]);
    group_barrier(g.bar, P);
    // every workgroup has read hist1 before arriving here: clear its share
    for (int b = (int)(part * NT) + t; b < HIST_BINS; b += (int)(P * NT)) st_agent(&g.hist1[b], 0u);
    find_bin_global<NT>(g.hist2, need2, sh.scratch, sh.found);
  } else {
    find_bin<NT, HIST_BINS>(sh.hist, need2, sh.scratch, sh.found);
  }
  const uint32_t b2 = sh.found[0];
  const uint32_t need3 = need2 - sh.found[1];
  const uint32_t p24 = (b1 << 12) | b2;
  __syncthreads();

  // ---- pass 3: bits 6..0 of keys whose bits 30..7 equal p24, and the count
  // of keys with a larger 24-bit prefix
  zero_lds<NT>(sh.hist, LAST_BINS);
  __syncthreads();
  uint32_t gtp = 0;
  if (listed) {
    for (uint32_t i = (uint32_t)lane_id(); i < ccount; i += WAVE) {
      const uint32_t kk = cand[i];
      if ((kk >> 7) == p24) atomicAdd(&sh.hist[kk & 0x7Fu], 1u);
      gtp += ((kk >> 7) > p24) ? 1u : 0u;
    }
    gtp += gt1;
  } else {
    count_digits<NT, VPT>(key, nv, 7, p24, 0, 0x7Fu, sh.hist);
#pragma unroll
    for (int v = 0; v < VPT; ++v)
      if (v < nv && (key[v] >> 7) > p24) ++gtp;
  }
  const uint32_t gtp_wg = block_sum<NT>(gtp, sh.scratch);   // contains barriers
  uint32_t* hall = sh.hist + HIST_BINS - 2 * LAST_BINS;     // [LAST_BINS] whole segment
  uint32_t* hbef = sh.hist + HIST_BINS - LAST_BINS;         // [LAST_BINS] lower workgroups
  uint32_t gtpb = 0;     // larger-prefix keys in lower workgroups
  if (P > 1) {
    const uint32_t pitch = slot_pitch(P);
    for (int b = t; b < LAST_BINS; b += NT) st_agent(&g.slots[(uint64_t)b * pitch + part], sh.hist[b]);
    if (t == 0) st_agent(&g.slots[(uint64_t)LAST_BINS * pitch + part], gtp_wg);
    group_barrier(g.bar, P);
    for (int b = (int)(part * NT) + t; b < HIST_BINS; b += (int)(P * NT)) st_agent(&g.hist2[b], 0u);
    // gather: row `bin` holds the bin's count of every workgroup; NT/128
    // thread sets split each row, reading it in 8-byte pairs (padding reads 0)
    constexpr int SETS = NT / LAST_BINS;
    const int bin = t % LAST_BINS, set = t / LAST_BINS;
    const uint32_t per = pitch / SETS;          // even: pitch is a multiple of 8
    const uint64_t* row = reinterpret_cast<const uint64_t*>(g.slots + (uint64_t)bin * pitch + set * per);
    uint32_t a_all = 0, a_bef = 0;
    for (uint32_t q = 0; q < per / 2; ++q) {
      const uint64_t pr = ld_agent64(row + q);
      const uint32_t j = set * per + 2 * q;
      const uint32_t lo = (uint32_t)pr, hi = (uint32_t)(pr >> 32);
      a_all += lo + hi;
      a_bef += (j < part ? lo : 0u) + (j + 1 < part ? hi : 0u);
    }
    // larger-prefix counts of the lower workgroups, in pairs as well
    uint32_t g_own = 0;
    {
      const uint64_t* grow = reinterpret_cast<const uint64_t*>(g.slots + (uint64_t)LAST_BINS * pitch);
      for (uint32_t q = (uint32_t)t; 2 * q < part; q += NT) {
        const uint64_t pr = ld_agent64(grow + q);
        g_own += (uint32_t)pr + ((2 * q + 1 < part) ? (uint32_t)(pr >> 32) : 0u);
      }
    }
    __syncthreads();
    uint32_t* red = sh.hist;   // [SETS][2][LAST_BINS] partial sums (bins 0..1023, free now)
    red[(set * 2) * LAST_BINS + bin] = a_all;
    red[(set * 2 + 1) * LAST_BINS + bin] = a_bef;
    __syncthreads();
    if (t < LAST_BINS) {
      uint32_t s_all = 0, s_bef = 0;
#pragma unroll
      for (int q = 0; q < SETS; ++q) { s_all += red[(q * 2) * LAST_BINS + t]; s_bef += red[(q * 2 + 1) * LAST_BINS + t]; }
      hall[t] = s_all;
      hbef[t] = s_bef;
    }
    gtpb = block_sum<NT>(g_own, sh.scratch);
  } else {
    if (t < LAST_BINS) { hall[t] = sh.hist[t]; hbef[t] = 0u; }
  }
  __syncthreads();
  find_bin<NT, LAST_BINS>(hall, need3, sh.scratch, sh.found);
  const uint32_t d3 = sh.found[0];
  res.T = (p24 << 7) | d3;
  res.r = need3 - sh.found[1];
  if (P > 1) {
    // keys > T before us: larger prefix, or same prefix with a larger last digit
    const uint32_t gt_digit = (t < LAST_BINS && (uint32_t)t > d3) ? hbef[t] : 0u;
    res.gt_before = gtpb + block_sum<NT>(gt_digit, sh.scratch);
    res.eq_before = hbef[d3 & (LAST_BINS - 1)];
  } else {
    res.gt_before = 0u;
    res.eq_before = 0u;
  }
  return res;
}

// Exact threshold for a segment held entirely by one wavefront (NT == 64).
template <int VPT>
__device__ __forceinline__ SelResult bitwise_select(const uint32_t (&key)[VPT], int nv, uint32_t k) {
  uint32_t T = 0u;
  for (int bit = 30; bit >= 0; --bit) {
    const uint32_t cand = T | (1u << bit);
    uint32_t cnt = 0;
#pragma unroll
    for (int v = 0; v < VPT; ++v) cnt += (uint32_t)__popcll(__ballot(v < nv && key[v] >= cand));
    if (cnt >= k) T = cand;
  }
  uint32_t gt = 0;
#pragma unroll
  for (int v = 0; v < VPT; ++v) gt += (uint32_t)__popcll(__ballot(v < nv && key[v] > T));
  SelResult res;
  res.T = T;
  res.r = k - gt;
  res.gt_before = 0u;
  res.eq_before = 0u;
  return res;
}

// Per-thread output placement after selection.  Entries of a thread are
// contiguous and in index order, threads in index order, workgroups of a
// segment in index order.
struct Placement {
  uint32_t pos;        // payload slot of this thread's first kept entry
  uint32_t tie_keep;   // how many of this thread's ties are kept
  uint32_t wg_first;   // payload slot of the workgroup's first kept entry
  uint32_t wg_count;   // entries the workgroup keeps
};

template <int NT, int VPT>
__device__ __forceinline__ Placement place(const uint32_t (&key)[VPT], int nv, const SelResult& s,
                                           uint32_t* scratch) {
  uint32_t gt = 0, eq = 0;
#pragma unroll
  for (int v = 0; v < VPT; ++v) {
    if (v < nv) { gt += key[v] > s.T; eq += key[v] == s.T; }
  }
  // both counts stay below 2^16 per workgroup (NT * VPT <= 32768)
  uint32_t tot;
  const uint32_t ex = block_excl_scan<NT>(gt | (eq << 16), scratch, tot);
  const uint32_t gt_ex = ex & 0xFFFFu, eq_ex = ex >> 16, eq_wg = tot >> 16;
  const uint32_t quota_wg = min(sat_sub(s.r, s.eq_before), eq_wg);
  const uint32_t mine = min(sat_sub(quota_wg, eq_ex), eq);
  Placement p;
  p.wg_first = s.gt_before + min(s.eq_before, s.r);
  p.wg_count = (tot & 0xFFFFu) + quota_wg;
  p.pos = p.wg_first + gt_ex + min(eq_ex, quota_wg);
  p.tie_keep = mine;
  return p;
}

}  // namespace tc
