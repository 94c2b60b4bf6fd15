// tc_select.hpp -- exact TopK threshold selection on register-resident keys.
//
// TopK (Sec. 2.3 of the paper) keeps the k entries of largest magnitude.  On
// the device the magnitude is the 31-bit key of mag_key(); the k-th largest
// key T and the tie quota r = k - #(key > T) define the kept set:
//   key > T, or key == T and the entry is among the r lowest-index ties.
//
// Shared pieces: bin search over histograms (in LDS or merged in device
// memory), and the one-wavefront strategy for short segments (a token row):
// a radix select over 8-bit digits with a wavefront-private histogram.  The
// several-workgroup strategy is in tc_group.hpp.
#pragma once

#include "tc_device.hpp"

namespace tc {

constexpr int HIST_BINS = 4096;   // 12-bit digits for the first two passes
constexpr int LAST_BINS = 128;    // 7-bit digit for the last pass
constexpr int SLOT_ROWS = LAST_BINS + 1;   // per-workgroup slot: 128 bins + larger-prefix count

// slot rows are laid out transposed, [row][workgroup], each row padded to a
// multiple of 8 workgroups so that readers can take them in 8-byte pairs
__host__ __device__ constexpr uint32_t slot_pitch(uint32_t P) { return (P + 7u) & ~7u; }

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

// ... with a small histogram in LDS, searched by the first wavefront alone
// (every thread calls; all meet at the closing barrier)
template <int NB>
__device__ __forceinline__ void find_bin_wave(const uint32_t* h, uint32_t need, uint32_t* found) {
  static_assert(NB % WAVE == 0, "whole bins per lane");
  constexpr int BPL = NB / WAVE;
  if (threadIdx.x < WAVE) {
    const int l = lane_id();
    uint32_t loc[BPL], sum = 0;
#pragma unroll
    for (int i = 0; i < BPL; ++i) {
      loc[i] = h[l * BPL + i];
      sum += loc[i];
    }
    const uint32_t incl = wave_incl_scan(sum);
    uint32_t acc = (uint32_t)__builtin_amdgcn_readlane((int)incl, WAVE - 1) - incl;   // bins of higher lanes
    if (acc < need && need <= acc + sum) {
#pragma unroll
      for (int i = BPL - 1; i >= 0; --i) {
        if (acc + loc[i] >= need) { found[0] = (uint32_t)(l * BPL + i); found[1] = acc; break; }
        acc += loc[i];
      }
    }
  }
  __syncthreads();
}

template <int NT>
__device__ __forceinline__ void zero_lds(uint32_t* h, int n) {
  for (int b = (int)threadIdx.x; b < n; b += NT) h[b] = 0u;
}

// Exact threshold for a segment held entirely by one wavefront (NT == 64):
// radix select over 8-bit digits of the key from bit 23 down, then its last
// 7 bits, with 256-bin histograms in LDS private to the wavefront (`hist`,
// 16-byte aligned, RADIX_CP * RADIX_HS words); each digit is found with one
// wavefront scan (lane l owns bins 4l..4l+3).
//  - The first digit is the exponent.  With at most 15 keys per lane it is
//    counted in registers first: a 4-bit counter per lane for each of the
//    eight digits at and below the segment's largest, summed over the
//    wavefront in four words.  Only when T's digit lies further down does
//    the histogram pass run.
//  - In that pass the exponent takes few values, so the lanes count in
//    RADIX_CP copies (lane mod RADIX_CP), RADIX_HS words apart: an odd
//    number of 4-word bank groups, so that one bin's copies sit in distinct
//    LDS banks.
//  - Once the chosen bin must give up only its largest key (one more
//    needed) or all of its keys, the rest of T is that largest or smallest
//    key, found by one wavefront reduction instead of the remaining passes
//    (after two digits a row's bin holds about one key).
constexpr int RADIX_CP = 4;
constexpr int RADIX_HS = 260;
template <int VPT>
__device__ __forceinline__ SelResult wave_radix_select(const uint32_t (&key)[VPT], int nv, uint32_t k,
                                                       uint32_t* hist) {
  const uint32_t lane = (uint32_t)lane_id();
  uint32_t prefix = 0u, need = k, pbits = 0u;
  // T from the keys under `prefix` (pbits bits): their largest (one copy
  // kept) or their smallest (all copies kept)
  auto settle = [&](bool top) {
    const uint32_t sh = 31u - pbits;
    uint32_t best = top ? 0u : 0xFFFFFFFFu;
#pragma unroll
    for (int i = 0; i < VPT; ++i)
      if (i < nv && (key[i] >> sh) == prefix) best = top ? max(best, key[i]) : min(best, key[i]);
    SelResult res;
    res.T = top ? wave_uminmax<true>(best) : wave_uminmax<false>(best);
    uint32_t eq = 0u;
    if (!top) {
#pragma unroll
      for (int i = 0; i < VPT; ++i) eq += (i < nv && key[i] == res.T) ? 1u : 0u;
    }
    res.r = top ? 1u : wave_sum(eq);
    res.gt_before = 0u;
    res.eq_before = 0u;
    return res;
  };
  int first = 0;   // digit passes already done
  if constexpr (VPT <= 15) {
    uint32_t dm = 0u;
#pragma unroll
    for (int i = 0; i < VPT; ++i)
      if (i < nv) dm = max(dm, key[i] >> 23);
    dm = wave_uminmax<true>(dm);
    uint32_t w = 0u;   // nibble o: keys of digit dm - o
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      const uint32_t off = dm - (key[i] >> 23);
      w += (i < nv && off < 8u) ? (1u << (off << 2)) : 0u;
    }
    // widened to 16-bit fields before the sums: words hold digits (0, 4),
    // (2, 6), (1, 5), (3, 7)
    const uint32_t ev = w & 0x0F0F0F0Fu, od = (w >> 4) & 0x0F0F0F0Fu;
    const uint32_t s04 = wave_sum(ev & 0x00FF00FFu), s26 = wave_sum((ev >> 8) & 0x00FF00FFu);
    const uint32_t s15 = wave_sum(od & 0x00FF00FFu), s37 = wave_sum((od >> 8) & 0x00FF00FFu);
    const uint32_t c8[8] = {s04 & 0xFFFFu, s15 & 0xFFFFu, s26 & 0xFFFFu, s37 & 0xFFFFu,
                            s04 >> 16,     s15 >> 16,     s26 >> 16,     s37 >> 16};
    uint32_t acc = 0u, cnt = 0u;
#pragma unroll
    for (int o = 0; o < 8; ++o) {
      if (first == 0 && acc < need && need <= acc + c8[o]) {
        first = 1;
        prefix = dm - (uint32_t)o;
        need -= acc;
        cnt = c8[o];
      }
      acc += c8[o];
    }
    if (first) {
      pbits = 8u;
      if (need == 1u || need == cnt) return settle(need == 1u);
    }
  }
#pragma unroll
  for (int pass = 0; pass < 4; ++pass) {
    if (pass < first) continue;
    const uint32_t width = (pass < 3) ? 8u : 7u;
    const uint32_t shift = 31u - pbits - width;
    constexpr int CP = RADIX_CP;
#pragma unroll
    for (int c = 0; c < (pass == 0 ? CP : 1); ++c)
      reinterpret_cast<u32x4*>(hist)[c * (RADIX_HS / 4) + lane] = u32x4{0u, 0u, 0u, 0u};
    __syncthreads();
    const uint32_t base = (pass == 0) ? (lane % CP) * (uint32_t)RADIX_HS : 0u;
#pragma unroll
    for (int i = 0; i < VPT; ++i)
      if (i < nv && (key[i] >> (shift + width)) == prefix)
        atomicAdd(&hist[base + ((key[i] >> shift) & ((1u << width) - 1u))], 1u);
    __syncthreads();
    u32x4 h = reinterpret_cast<const u32x4*>(hist)[lane];
    if (pass == 0) {
#pragma unroll
      for (int c = 1; c < CP; ++c) {
        const u32x4 hc = reinterpret_cast<const u32x4*>(hist)[c * (RADIX_HS / 4) + lane];
        h = h + hc;
      }
    }
    const uint32_t sum = h[0] + h[1] + h[2] + h[3];
    const uint32_t incl = wave_incl_scan(sum);
    uint32_t acc = (uint32_t)__builtin_amdgcn_readlane((int)incl, WAVE - 1) - incl;   // bins of higher lanes
    uint32_t d = 0u, cnt = 0u;
    const bool here = acc < need && need <= acc + sum;
    if (here) {
#pragma unroll
      for (int c = 3; c >= 0; --c) {
        if (acc + h[c] >= need) { d = 4u * lane + (uint32_t)c; cnt = h[c]; break; }
        acc += h[c];
      }
    }
    const int src = __builtin_ctzll(__ballot(here));
    d = (uint32_t)__builtin_amdgcn_readlane((int)d, src);
    acc = (uint32_t)__builtin_amdgcn_readlane((int)acc, src);
    cnt = (uint32_t)__builtin_amdgcn_readlane((int)cnt, src);
    prefix = (prefix << width) | d;
    need -= acc;
    pbits += width;
    __syncthreads();
    if (pass < 3 && (need == 1u || need == cnt)) return settle(need == 1u);
  }
  SelResult res;
  res.T = prefix;
  res.r = need;
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
