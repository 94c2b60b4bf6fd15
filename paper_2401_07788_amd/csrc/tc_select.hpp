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
constexpr int SLOT_WORDS = 132;   // per-workgroup slot: 128 bins + larger-prefix count (+pad)

// device memory owned by one group of P workgroups (inside the caller's
// workspace, zero-filled before first use and left zero-filled on exit)
struct GroupMem {
  uint32_t* bar;     // [2] barrier count / sense
  uint32_t* hist1;   // [HIST_BINS]
  uint32_t* hist2;   // [HIST_BINS]
  uint32_t* slots;   // [P][SLOT_WORDS]
};

// words of workspace per group (barrier padded to 64 words)
__host__ __device__ constexpr uint64_t group_mem_words(uint32_t P) {
  return 64u + 2u * HIST_BINS + (uint64_t)P * SLOT_WORDS;
}

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
  uint32_t scratch[NT / WAVE + 2];
  uint32_t found[2];          // bin, count above it
};

struct SelResult {
  uint32_t T;          // threshold key (0xFFFFFFFF when k == 0: nothing kept)
  uint32_t r;          // ties at T to keep over the whole segment
  uint32_t gt_before;  // keys > T in lower-indexed workgroups of the segment
  uint32_t eq_before;  // keys == T in lower-indexed workgroups of the segment
};

// Find the bin b of h[0..NB) with  sum_{c > b} h[c] < need <= sum_{c >= b} h[c]
// (1 <= need <= sum h).  Writes (b, sum_{c > b} h[c]) to found[].
template <int NT, int NB>
__device__ __forceinline__ void find_bin(const uint32_t* h, uint32_t need, uint32_t* scratch,
                                         uint32_t* found) {
  constexpr int BPT = (NB + NT - 1) / NT;
  const int t = (int)threadIdx.x;
  uint32_t loc[BPT];
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    const int b = t * BPT + i;
    loc[i] = (b < NB) ? h[b] : 0u;
    sum += loc[i];
  }
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
  SelResult res;
  // ---- pass 1: bits 30..19 of all keys
  zero_lds<NT>(sh.hist, HIST_BINS);
  __syncthreads();
  count_digits<NT, VPT>(key, nv, 31, 0u, 19, 0xFFFu, sh.hist);
  __syncthreads();
  if (P > 1) {
    for (int b = (int)threadIdx.x; b < HIST_BINS; b += NT)
      if (sh.hist[b]) add_agent(&g.hist1[b], sh.hist[b]);
    group_barrier(g.bar, P);
    for (int b = (int)threadIdx.x; b < HIST_BINS; b += NT) sh.hist[b] = ld_agent(&g.hist1[b]);
    __syncthreads();
  }
  find_bin<NT, HIST_BINS>(sh.hist, k, sh.scratch, sh.found);
  const uint32_t b1 = sh.found[0];
  const uint32_t need2 = k - sh.found[1];
  __syncthreads();

  // ---- pass 2: bits 18..7 of keys whose bits 30..19 equal b1
  zero_lds<NT>(sh.hist, HIST_BINS);
  __syncthreads();
  count_digits<NT, VPT>(key, nv, 19, b1, 7, 0xFFFu, sh.hist);
  __syncthreads();
  if (P > 1) {
    for (int b = (int)threadIdx.x; b < HIST_BINS; b += NT)
      if (sh.hist[b]) add_agent(&g.hist2[b], sh.hist[b]);
    group_barrier(g.bar, P);
    // every workgroup has read hist1 before arriving here: clear its share
    for (int b = (int)(part * NT + threadIdx.x); b < HIST_BINS; b += (int)(P * NT)) st_agent(&g.hist1[b], 0u);
    for (int b = (int)threadIdx.x; b < HIST_BINS; b += NT) sh.hist[b] = ld_agent(&g.hist2[b]);
    __syncthreads();
  }
  find_bin<NT, HIST_BINS>(sh.hist, need2, sh.scratch, sh.found);
  const uint32_t b2 = sh.found[0];
  const uint32_t need3 = need2 - sh.found[1];
  const uint32_t p24 = (b1 << 12) | b2;
  __syncthreads();

  // ---- pass 3: bits 6..0 of keys whose bits 30..7 equal p24, and the count
  // of keys with a larger 24-bit prefix
  zero_lds<NT>(sh.hist, LAST_BINS);
  __syncthreads();
  count_digits<NT, VPT>(key, nv, 7, p24, 0, 0x7Fu, sh.hist);
  uint32_t gtp = 0;
#pragma unroll
  for (int v = 0; v < VPT; ++v)
    if (v < nv && (key[v] >> 7) > p24) ++gtp;
  const uint32_t gtp_wg = block_sum<NT>(gtp, sh.scratch);   // contains barriers
  if (P > 1) {
    uint32_t* mine = g.slots + (uint64_t)part * SLOT_WORDS;
    for (int b = (int)threadIdx.x; b < LAST_BINS; b += NT) st_agent(&mine[b], sh.hist[b]);
    if (threadIdx.x == 0) st_agent(&mine[LAST_BINS], gtp_wg);
    group_barrier(g.bar, P);
    for (int b = (int)(part * NT + threadIdx.x); b < HIST_BINS; b += (int)(P * NT)) st_agent(&g.hist2[b], 0u);
  }
  // gather: global last-digit histogram, and the part that lies before us
  uint32_t hb = 0;       // this thread's bin, summed over lower workgroups
  uint32_t gtpb = 0;     // larger-prefix keys in lower workgroups (thread 0)
  const int t = (int)threadIdx.x;
  if (P > 1) {
    if (t < LAST_BINS) {
      uint32_t hall = 0;
      for (uint32_t j = 0; j < P; ++j) {
        const uint32_t c = ld_agent(&g.slots[(uint64_t)j * SLOT_WORDS + t]);
        hall += c;
        if (j < part) hb += c;
      }
      sh.hist[HIST_BINS - LAST_BINS + t] = hall;
    }
    if (t == LAST_BINS % NT) {   // a thread other than those above when NT > 128
      for (uint32_t j = 0; j < part; ++j) gtpb += ld_agent(&g.slots[(uint64_t)j * SLOT_WORDS + LAST_BINS]);
    }
  } else {
    if (t < LAST_BINS) sh.hist[HIST_BINS - LAST_BINS + t] = sh.hist[t];
  }
  __syncthreads();
  find_bin<NT, LAST_BINS>(sh.hist + (HIST_BINS - LAST_BINS), need3, sh.scratch, sh.found);
  const uint32_t d3 = sh.found[0];
  res.T = (p24 << 7) | d3;
  res.r = need3 - sh.found[1];
  if (P > 1) {
    // keys > T before us: larger prefix, or same prefix with a larger last digit
    const uint32_t gt_digit = (t < LAST_BINS && (uint32_t)t > d3) ? hb : 0u;
    const uint32_t eq_digit = (t < LAST_BINS && (uint32_t)t == d3) ? hb : 0u;
    const uint32_t s1 = block_sum<NT>(gt_digit + gtpb, sh.scratch);
    const uint32_t s2 = block_sum<NT>(eq_digit, sh.scratch);
    res.gt_before = s1;
    res.eq_before = s2;
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
  p.pos = s.gt_before + min(s.eq_before, s.r) + gt_ex + min(eq_ex, quota_wg);
  p.tie_keep = mine;
  return p;
}

}  // namespace tc
