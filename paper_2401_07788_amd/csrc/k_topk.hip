// k_topk.hip -- the sender side of TopK (Sec. 2.3), with error feedback
// (Sec. 2.4) or AQ-SGD (Sec. 2.5) fused around it.
//
// One selection, three producers / epilogues:
//   PLAIN : v = x                                  -> payload
//   EF    : v = x + e                              -> payload, e <- v - r
//           r = what the receiver gets: wire(v) at kept entries, +0 elsewhere
//   AQSGD : v = a - m[id]                          -> payload, m[id][kept] += wire(v)
// and, in the LDS engine only, the two selections of EF-mixed (Sec. 2.4):
//   EFMIX : TopK(x) and TopK(e) over halves of the budget -> two payloads,
//           one workgroup each (they are independent); the residual
//           e <- (x - r_x) + (e - r_e) is k_efmix_resid's (k_scatter.hip)
// The segment (a sample, a token row, a whole example) stays in registers or
// LDS for the whole kernel: inputs are read once, the selection works on
// registers and LDS, and the outputs are written once.
//
// Three engines:
//   k_topk_row : one wavefront per segment of up to 2048 elements (token
//                rows); radix select over 8-bit digits with a wavefront-
//                private LDS histogram, one wavefront scan per digit.
//   k_topk_lds : one 1024-thread workgroup per segment of up to 32,768
//                elements (per-sample tensors), the segment held in LDS.
//   k_topk_grp : P workgroups of 512 threads per segment (long samples,
//                examples); striped register layout, two cross-workgroup
//                exchanges (tc_group.hpp), payload staged in LDS and written
//                in index order with full-line stores.
#include <algorithm>
#include <type_traits>

#include "tc_group.hpp"
#include "tc_internal.hpp"

namespace tc {

// Workgroup -> (group, part).  Workgroups are dealt round-robin to the 8 XCDs;
// when the grid allows, the P workgroups of a group are taken from one XCD so
// that the group's cross-workgroup traffic stays behind one L2.
__device__ __forceinline__ void map_wg(uint32_t wg, uint32_t grid, uint32_t P, uint32_t& group,
                                       uint32_t& part) {
  if (P > 1 && grid % (8u * P) == 0u) {
    const uint32_t xcd = wg & 7u, q = wg >> 3;
    group = xcd + 8u * (q / P);
    part = q % P;
  } else {
    group = wg / P;
    part = wg % P;
  }
}

// ------------------------------------------------------------- row engine
template <typename InT, int SEL, int VPT>
__global__ __launch_bounds__(WAVE) void k_topk_row(TopkArgs a) {
  using R = typename Elem<InT>::raw;
  __shared__ uint32_t scratch[2];
  __shared__ __attribute__((aligned(16))) uint32_t hist[RADIX_CP * RADIX_HS];
  for (uint64_t seg = blockIdx.x; seg < a.n_seg; seg += gridDim.x) {
    const uint64_t c0 = (uint64_t)threadIdx.x * VPT;
    const int nv = (int)min((uint64_t)VPT, sat_sub(a.L, c0));

    // ---- producer: the vector to compress, in binary32
    float v[VPT];
    R mr[VPT];                 // AQSGD: the buffer row, kept for the update
    uint64_t mrow = 0;
    if constexpr (SEL == SEL_AQSGD) {
      const int64_t id = load_uniform(a.ids + seg);
      if (id < 0 || (uint64_t)id >= a.n_samples) {
        if (threadIdx.x == 0) raise_error(KERR_BAD_ID);
        continue;
      }
      mrow = (uint64_t)id * a.L;
    }
    {
      R xr[VPT];
      const uint64_t off = seg * a.L + c0;
      if (nv > 0) load_run_partial<R, VPT, true>((const R*)a.x + off, nv, R{}, xr);
      if constexpr (SEL == SEL_EF) {
        float er[VPT];
        if (nv > 0) load_run_partial<float, VPT, true>(a.e + off, nv, 0.0f, er);
#pragma unroll
        for (int i = 0; i < VPT; ++i) v[i] = (i < nv) ? Elem<InT>::up(xr[i]) + er[i] : 0.0f;
      } else if constexpr (SEL == SEL_AQSGD) {
        if (nv > 0) load_run_partial<R, VPT, true>((const R*)a.m + mrow + c0, nv, R{}, mr);
#pragma unroll
        for (int i = 0; i < VPT; ++i) v[i] = (i < nv) ? Elem<InT>::up(xr[i]) - Elem<InT>::up(mr[i]) : 0.0f;
      } else {
#pragma unroll
        for (int i = 0; i < VPT; ++i) v[i] = (i < nv) ? Elem<InT>::up(xr[i]) : 0.0f;
      }
    }
    uint32_t key[VPT];
#pragma unroll
    for (int i = 0; i < VPT; ++i) key[i] = mag_key(v[i]);

    SelResult sr;
    if (a.k == 0) { sr.T = 0xFFFFFFFFu; sr.r = 0; sr.gt_before = 0; sr.eq_before = 0; }
    else sr = wave_radix_select<VPT>(key, nv, (uint32_t)a.k, hist);
    const Placement pl = place<WAVE, VPT>(key, nv, sr, scratch);

    uint32_t* idx = a.idx + seg * a.k;
    R* val = (R*)a.val + seg * a.k;
    uint32_t pos = pl.pos, ties = 0;
    float eo[VPT];
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
      bool kept = false;
      if (i < nv) {
        const bool tie = key[i] == sr.T;
        kept = key[i] > sr.T || (tie && ties < pl.tie_keep);
        ties += tie ? 1u : 0u;
        if (kept) {
          const R w = Elem<InT>::down(v[i]);
          if (pos < a.k) { idx[pos] = (uint32_t)(c0 + i); val[pos] = w; }
          else raise_error(KERR_INTERNAL);
          ++pos;
          if constexpr (SEL == SEL_AQSGD) mr[i] = Elem<InT>::down(Elem<InT>::up(mr[i]) + Elem<InT>::up(w));
        }
      }
      if constexpr (SEL == SEL_EF) eo[i] = v[i] - (kept ? through<InT>(v[i]) : 0.0f);
    }
    if constexpr (SEL == SEL_EF) {
      if (nv > 0) store_run_partial<float, VPT, true>(a.e + seg * a.L + c0, nv, eo);
    }
    if constexpr (SEL == SEL_AQSGD) {
      if (nv > 0 && a.k > 0) store_run_partial<R, VPT, false>((R*)a.m + mrow + c0, nv, mr);
    }
    if (a.blk && threadIdx.x == 0) {
      // a wavefront segment is shorter than one block
      uint32_t* bt = a.blk + seg * (n_blocks(a.L) + 1);
      bt[0] = 0;
      bt[n_blocks(a.L)] = (uint32_t)a.k;
    }
  }
}

// ----------------------------------------------------------- group engine
// LDS: the selection's histogram and candidate list, then (after the
// selection) the workgroup's payload entries, staged so that they leave in
// index order with full-line stores; WAVE extra entries are per-lane dummy
// slots for the entries a lane does not keep.
template <uint32_t CH, typename Raw>
union GrpShared {
  GrpSelShared<grp_local_cap(CH)> sel;
  struct {
    uint32_t idx[CH + WAVE];
    Raw val[CH + WAVE];
  } st;
};

// one 16-byte run of E elements (full, 16-byte aligned)
template <typename Raw, int E, bool STREAM>
__device__ __forceinline__ void load16(const Raw* p, Raw (&out)[E]) {
  static_assert(E * sizeof(Raw) == 16, "one 16-byte access");
  const u32x4 w = vload<STREAM>(reinterpret_cast<const u32x4*>(p));
  __builtin_memcpy(out, &w, 16);
}
// one 16-byte run at base + off when `in`, else the run at base (one the
// caller knows to be in bounds, and discards): the address is a select, so
// that no branch stands between the loads
template <typename Raw, int E, bool STREAM>
__device__ __forceinline__ void load16_in(const Raw* base, uint32_t off, bool in, Raw (&out)[E]) {
  load16<Raw, E, STREAM>(base + (in ? off : 0u), out);
}
template <typename Raw, int E, bool STREAM>
__device__ __forceinline__ void store16(Raw* p, const Raw (&in)[E]) {
  static_assert(E * sizeof(Raw) == 16, "one 16-byte access");
  u32x4 w;
  __builtin_memcpy(&w, in, 16);
  vstore<STREAM>(reinterpret_cast<u32x4*>(p), w);
}

// Copy n staged entries to dst, leaving some out: rem[0..nr) (nr <= WAVE)
// holds the staged position of each left-out entry less the number of
// left-out entries before it (non-decreasing), so that output entry o comes
// from staged position o + #{i : rem[i] <= o}.  A wavefront writes 64
// consecutive 16-byte pieces at a time; the few left-out entries that fall
// among them are counted with ballots and one loop over that set.
template <int NT, typename T>
__device__ __forceinline__ void copy_lds_skip(T* __restrict__ dst, const T* src, uint32_t n, const uint32_t* rem,
                                              uint32_t nr) {
  constexpr uint32_t PER = 16 / sizeof(T);
  const uint32_t lane = (uint32_t)lane_id(), wv = threadIdx.x / WAVE;
  const uint32_t rv = (lane < nr) ? rem[lane] : ~0u;     // lane i holds rem[i]
  const uint32_t mis = (uint32_t)(((uintptr_t)dst / sizeof(T)) % PER);
  const uint32_t head = min(n, (PER - mis) % PER);
  const uint32_t body = (n - head) / PER;
  const uint32_t done = head + body * PER;
  // the unaligned head and the tail (fewer than PER entries each): one
  // entry per lane, by wavefronts 0 and 1
  if (wv < 2) {
    const uint32_t o0 = (wv == 0) ? 0u : done, cnt = (wv == 0) ? head : n - done;
    uint32_t d = (uint32_t)__popcll(__ballot(rv < o0));
    uint64_t in = __ballot(rv >= o0 && rv < o0 + PER);
    while (in) {
      const int i = __builtin_ctzll(in);
      in &= in - 1;
      d += ((uint32_t)__builtin_amdgcn_readlane((int)rv, i) <= o0 + lane) ? 1u : 0u;
    }
    if (lane < cnt) dst[o0 + lane] = src[o0 + lane + d];
  }
  for (uint32_t base = wv * WAVE; base < body; base += NT) {
    const uint32_t A = head + base * PER;              // the wavefront's first output
    const uint32_t o = A + lane * PER;                 // this lane's first output
    const uint32_t d0 = (uint32_t)__popcll(__ballot(rv <= A));
    uint64_t in = __ballot(rv > A && rv < A + WAVE * PER);
    uint32_t d[PER];
#pragma unroll
    for (uint32_t e = 0; e < PER; ++e) d[e] = d0;
    while (in) {
      const int i = __builtin_ctzll(in);
      in &= in - 1;
      const uint32_t r = (uint32_t)__builtin_amdgcn_readlane((int)rv, i);
#pragma unroll
      for (uint32_t e = 0; e < PER; ++e) d[e] += (r <= o + e) ? 1u : 0u;
    }
    if (base + lane < body) {
      T tmp[PER];
#pragma unroll
      for (uint32_t e = 0; e < PER; ++e) tmp[e] = src[o + e + d[e]];
      u32x4 w;
      __builtin_memcpy(&w, tmp, 16);
      vstore<true>(reinterpret_cast<u32x4*>(dst + o), w);
    }
  }
}

// The same for the index and value lists together, four entries per lane
// and piece, when both destinations sit alike against their 4-entry pieces
// (the usual case); otherwise one list after the other.
template <int NT, typename T>
__device__ __forceinline__ void copy_lds_skip2(uint32_t* __restrict__ di, T* __restrict__ dv, const uint32_t* si,
                                               const T* sv, uint32_t n, const uint32_t* rem, uint32_t nr) {
  constexpr uint32_t PER = 4;
  const uint32_t mis = (uint32_t)(((uintptr_t)di / 4u) % PER);
  if ((((uintptr_t)dv / sizeof(T)) % PER) != mis || ((uintptr_t)dv % sizeof(T)) != 0) {
    copy_lds_skip<NT>(di, si, n, rem, nr);
    copy_lds_skip<NT>(dv, sv, n, rem, nr);
    return;
  }
  const uint32_t lane = (uint32_t)lane_id(), wv = threadIdx.x / WAVE;
  const uint32_t rv = (lane < nr) ? rem[lane] : ~0u;     // lane i holds rem[i]
  const uint32_t head = min(n, (PER - mis) % PER);
  const uint32_t body = (n - head) / PER;
  const uint32_t done = head + body * PER;
  if (wv < 2) {
    const uint32_t o0 = (wv == 0) ? 0u : done, cnt = (wv == 0) ? head : n - done;
    uint32_t d = (uint32_t)__popcll(__ballot(rv < o0));
    uint64_t in = __ballot(rv >= o0 && rv < o0 + PER);
    while (in) {
      const int i = __builtin_ctzll(in);
      in &= in - 1;
      d += ((uint32_t)__builtin_amdgcn_readlane((int)rv, i) <= o0 + lane) ? 1u : 0u;
    }
    if (lane < cnt) {
      di[o0 + lane] = si[o0 + lane + d];
      dv[o0 + lane] = sv[o0 + lane + d];
    }
  }
  for (uint32_t base = wv * WAVE; base < body; base += NT) {
    const uint32_t A = head + base * PER;
    const uint32_t o = A + lane * PER;
    const uint32_t d0 = (uint32_t)__popcll(__ballot(rv <= A));
    uint64_t in = __ballot(rv > A && rv < A + WAVE * PER);
    uint32_t d[PER];
#pragma unroll
    for (uint32_t e = 0; e < PER; ++e) d[e] = d0;
    while (in) {
      const int i = __builtin_ctzll(in);
      in &= in - 1;
      const uint32_t r = (uint32_t)__builtin_amdgcn_readlane((int)rv, i);
#pragma unroll
      for (uint32_t e = 0; e < PER; ++e) d[e] += (r <= o + e) ? 1u : 0u;
    }
    if (base + lane < body) {
      uint32_t ti[PER];
      T tv[PER];
#pragma unroll
      for (uint32_t e = 0; e < PER; ++e) {
        ti[e] = si[o + e + d[e]];
        tv[e] = sv[o + e + d[e]];
      }
      u32x4 wi;
      __builtin_memcpy(&wi, ti, 16);
      vstore<true>(reinterpret_cast<u32x4*>(di + o), wi);
      if constexpr (sizeof(T) == 4) {
        u32x4 w;
        __builtin_memcpy(&w, tv, 16);
        vstore<true>(reinterpret_cast<u32x4*>(dv + o), w);
      } else {
        static_assert(sizeof(T) == 2, "16-bit or 32-bit values");
        u32x2 w;
        __builtin_memcpy(&w, tv, 8);
        vstore<true>(reinterpret_cast<u32x2*>(dv + o), w);
      }
    }
  }
}

// Exchange B with the payload and buffer work moved ahead (fine mode, 2 <= P
// <= REC_P_MAX).  The 16-bit prefix `pre` of T already divides the keys:
// those above it are kept whatever T is, those below are dropped, and only
// the few on it wait for exchange B.  Before the group's barrier: the keys on
// the prefix go into the record; then, while the other workgroups arrive,
// every entry above or on the prefix is staged in LDS in index order and the
// buffer rows are stored as if only the keys above the prefix were kept.
// After the barrier one wavefront decides the keys on the prefix and stores
// the buffer values of the kept ones; the others are left out of the staged
// list when it is copied out.  Returns
// false when a record overflowed: nothing decided, the buffer rows are then
// stored again by the caller.
template <typename InT, int SEL, int R>
__device__ __forceinline__ bool grp_early(const TopkArgs& a, bool vec, uint64_t seg, uint32_t P, uint32_t part,
                                          const GrpMem& gm,
                                          GrpShared<(uint32_t)GRP_NT * R * (16 / sizeof(typename Elem<InT>::raw)),
                                                    typename Elem<InT>::raw>& sh,
                                          GrpSmall& sm, GrpState& gs, const SelA& A,
                                          float (&v)[R][16 / sizeof(typename Elem<InT>::raw)], const int (&n)[R],
                                          uint64_t c0, typename Elem<InT>::raw* ms, float* es,
                                          const typename Elem<InT>::raw* mlds, bool exiting, uint32_t& ticket) {
  using Raw = typename Elem<InT>::raw;
  constexpr int NT = GRP_NT;
  constexpr int E = 16 / (int)sizeof(Raw);
  constexpr uint32_t CH = (uint32_t)NT * R * E;
  const int t = (int)threadIdx.x;
  const uint32_t dummy = (uint32_t)lane_id();
  const uint32_t pre = A.prefix;   // bits 30..15 of T

  // ---- per run: entries above or on the prefix, and on it (both < 2^16
  // per workgroup), scanned in index order; the thread's own ones as bit
  // masks (bit i: element i of the run)
  static_assert(E <= 8, "two 8-bit masks per run");
  if (t < (int)DIG_BINS) sm.red[t] = 0u;
  uint32_t pc[R], ex[R], tot[R], msk[R];
#pragma unroll
  for (int j = 0; j < R; ++j) {
    uint32_t mm = 0, cm = 0;
#pragma unroll
    for (int i = 0; i < E; ++i) {
      const uint32_t hi = mag_key(v[j][i]) >> 15;
      const uint32_t on = eq31(hi, pre);
      mm |= (gt31(hi, pre) | on) << i;
      cm |= on << i;
    }
    msk[j] = mm | (cm << 8);
    pc[j] = (uint32_t)__builtin_popcount(mm) | ((uint32_t)__builtin_popcount(cm) << 16);
  }
  block_excl_scan_multi<NT, R>(pc, ex, tot, sm.scratch);
  refresh(v);
  uint32_t mb[R], cb[R];      // the workgroup's staged entries / keys on the prefix in runs before j
  uint32_t m_all = 0, c_all = 0;
#pragma unroll
  for (int j = 0; j < R; ++j) {
    mb[j] = m_all;
    cb[j] = c_all;
    m_all += tot[j] & 0xFFFFu;
    c_all += tot[j] >> 16;
  }

  // ---- the keys on the prefix (a few per workgroup): record slot (index
  // order), their bits 14..7 into the digit counts, and what deciding them
  // later needs; a thread visits only the set bits of its masks
  uint32_t* my = gm.rec() + (uint64_t)part * REC_W;
#pragma unroll
  for (int j = 0; j < R; ++j) {
    uint32_t cm = msk[j] >> 8;
    if (cm) {
      uint32_t q = cb[j] + (ex[j] >> 16);
      const uint32_t sp0 = mb[j] + (ex[j] & 0xFFFFu), mm = msk[j] & 0xFFu;
      const uint32_t off = (uint32_t)(j * NT + t) * E;
      do {
        const uint32_t i = (uint32_t)__builtin_ctz(cm);
        cm &= cm - 1u;
        uint32_t kk = mag_key(v[j][0]);
#pragma unroll
        for (int ii = 1; ii < E; ++ii) kk = (i == (uint32_t)ii) ? mag_key(v[j][ii]) : kk;
        if (q < REC_KEYS) {
          st_agent(&my[2 + q], kk);
          sm.ckey[q] = kk;
          sm.coff[q] = off + i;
          sm.cpos[q] = sp0 + (uint32_t)__builtin_popcount(mm & ((1u << i) - 1u));
        }
        atomicAdd(&sm.red[(kk >> 7) & 0xFFu], 1u);
        ++q;
      } while (cm);
    }
  }
  __syncthreads();
  grp_publish_b<NT>(part, gm, sm, gs, m_all - c_all, c_all);
  refresh(v);

  // ---- while the group arrives: stage the entries above or on the prefix
  // and store the buffer rows with only the keys above it kept
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const uint32_t off = (uint32_t)(j * NT + t) * E;
    uint32_t sp = mb[j] + (ex[j] & 0xFFFFu);
    Raw mr[E];
    float eo[E];
    if constexpr (SEL == SEL_AQSGD) load16<Raw, E, false>(mlds + off, mr);
#pragma unroll
    for (int i = 0; i < E; ++i) {
      const uint32_t mayb = (msk[j] >> i) & 1u, cert = mayb & ~(msk[j] >> (8 + i));
      const Raw w = Elem<InT>::down(v[j][i]);
      const uint32_t slot = pick(mayb, sp, CH + dummy);
      sh.st.idx[slot] = (uint32_t)c0 + off + (uint32_t)i;
      sh.st.val[slot] = w;
      sp += mayb;
      if constexpr (SEL == SEL_AQSGD) {
        const Raw upd = Elem<InT>::down(Elem<InT>::up(mr[i]) + Elem<InT>::up(w));
        if constexpr (sizeof(Raw) == 4) mr[i] = __uint_as_float(pick(cert, __float_as_uint(upd), __float_as_uint(mr[i])));
        else mr[i] = (Raw)pick(cert, upd, mr[i]);
      }
      if constexpr (SEL == SEL_EF) eo[i] = v[j][i] - __uint_as_float(pick(cert, __float_as_uint(through<InT>(v[j][i])), 0u));
    }
    if (vec && n[j] == E) {
      if constexpr (SEL == SEL_EF) {
        store16<float, 4, E == 4>(es + off, *reinterpret_cast<float(*)[4]>(&eo[0]));
        if constexpr (E == 8) store16<float, 4, false>(es + off + 4, *reinterpret_cast<float(*)[4]>(&eo[4]));
      }
      if constexpr (SEL == SEL_AQSGD) store16<Raw, E, true>(ms + off, mr);
    } else if (n[j] > 0) {
      if constexpr (SEL == SEL_EF) store_run_partial<float, E, true>(es + off, n[j], eo);
      if constexpr (SEL == SEL_AQSGD) store_run_partial<Raw, E, true>(ms + off, n[j], mr);
    }
  }

  SelResult sr;
  const bool ok = grp_finish_b<NT>((uint32_t)a.k, P, part, gm, sm, gs, A, sr);
  refresh(v);
  if (!ok) return false;
  // every wavefront's buffer stores are complete before some of them are
  // overwritten from another wavefront below
  if (exiting) ticket = grp_exit_ticket(gm);
  else {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  grp_finish_b_lower<NT>(sm, sr);

  // ---- decide the keys on the prefix (at most REC_KEYS: one wavefront);
  // the kept ones get their buffer values
  if (t < WAVE) {
    const bool has = (uint32_t)t < c_all;
    const uint32_t key = has ? sm.ckey[t] : 0u;
    const bool tie = has && key == sr.T;
    const uint64_t tm = __ballot(tie);
    const uint32_t quota = min(sat_sub(sr.r, sr.eq_before), (uint32_t)__popcll(tm));   // ties this workgroup keeps
    const bool kept = (has && key > sr.T) || (tie && lanes_below(tm) < quota);
    const bool drop = has && !kept;
    const uint64_t km = __ballot(kept), dm = __ballot(drop);
    const uint32_t off = has ? sm.coff[t] : 0u;
    if constexpr (SEL != SEL_PLAIN) {
      if (kept) {
        // the value sent is the staged one; the key and its sign give the
        // exact difference back
        const Raw w = sh.st.val[sm.cpos[t]];
        if constexpr (SEL == SEL_AQSGD) {
          const Raw upd = Elem<InT>::down(Elem<InT>::up(mlds[off]) + Elem<InT>::up(w));
          ms[off] = upd;
        }
        if constexpr (SEL == SEL_EF) {
          const float x = __uint_as_float(key | (__float_as_uint(Elem<InT>::up(w)) & 0x80000000u));
          es[off] = x - Elem<InT>::up(w);
        }
      }
    }
    if (drop) sm.rem[lanes_below(dm)] = sm.cpos[t] - lanes_below(dm);
    const uint32_t run = has ? off / (uint32_t)(NT * E) : (uint32_t)R;
    uint32_t rb[R];
#pragma unroll
    for (int j = 0; j < R; ++j) rb[j] = (uint32_t)__popcll(__ballot(drop && run < (uint32_t)j));
    if (t == 0) {
      sm.misc[2] = (uint32_t)__popcll(dm);
      sm.misc[3] = (uint32_t)__popcll(km);
      // block table: kept entries below each block boundary this workgroup
      // covers (boundaries start runs)
      if (a.blk) {
        const uint32_t wg_first = sr.gt_before + min(sr.eq_before, sr.r);
        uint32_t* bt = a.blk + seg * (n_blocks(a.L) + 1);
#pragma unroll
        for (int j = 0; j < R; ++j) {
          const uint64_t B = c0 + (uint64_t)j * NT * E;
          if (B % BLOCK_LEN == 0 && B < a.L) bt[B / BLOCK_LEN] = wg_first + mb[j] - rb[j];
        }
        if (part == 0) bt[n_blocks(a.L)] = (uint32_t)a.k;
      }
    }
  }
  __syncthreads();

  // ---- the workgroup's run of the payload, in index order, coalesced
  const uint32_t n_drop = sm.misc[2];
  const uint32_t wg_count = (m_all - c_all) + sm.misc[3];
  const uint32_t wg_first = sr.gt_before + min(sr.eq_before, sr.r);
  uint32_t* idx = a.idx + seg * a.k;
  Raw* val = (Raw*)a.val + seg * a.k;
  if (wg_first + wg_count > a.k) {
    if (t == 0) raise_error(KERR_INTERNAL);
  } else {
    copy_lds_skip2<NT>(idx + wg_first, val + wg_first, sh.st.idx, sh.st.val, wg_count, sm.rem, n_drop);
  }
  return true;
}

// One segment on one workgroup of its group.  `vec`: every buffer is 16-byte
// aligned and segments start on 16-byte boundaries, so that whole runs move
// as single 16-byte accesses; a run cut by the segment's end (or any run
// without `vec`) goes element by element.
template <typename InT, int SEL, int R>
__device__ __forceinline__ void grp_segment(const TopkArgs& a, bool vec, uint64_t seg, uint32_t P,
                                            uint32_t part, const GrpMem& gm,
                                            GrpShared<(uint32_t)GRP_NT * R * (16 / sizeof(typename Elem<InT>::raw)),
                                                      typename Elem<InT>::raw>& sh,
                                            GrpSmall& sm, GrpState& gs, bool last_seg, bool& exited,
                                            typename Elem<InT>::raw* mlds) {
  using Raw = typename Elem<InT>::raw;
  constexpr int NT = GRP_NT;
  constexpr int E = 16 / (int)sizeof(Raw);
  constexpr uint32_t CH = (uint32_t)NT * R * E;
  const int t = (int)threadIdx.x;
  const uint32_t dummy = (uint32_t)lane_id();
  const uint64_t c0 = (uint64_t)part * CH;
  const Raw* xs = (const Raw*)a.x + seg * a.L + c0;
  float* es = (SEL == SEL_EF) ? a.e + seg * a.L + c0 : nullptr;

  // ---- producer: run j of this thread starts at chunk offset (j*NT + t)*E;
  // all loads are issued before any is used, the input's before the buffer
  // row's address (AQSGD: the example id) is waited for.  With every buffer
  // 16-byte aligned and L a multiple of E (vec), a run lies wholly inside or
  // wholly past the segment's end: one past it reads the chunk's first run
  // (in bounds, as c0 < L) and its values become +0 below, so that the loads
  // carry no branch (a branch per run that writes the same registers on
  // both sides makes each load wait for the one before).  Otherwise runs
  // load element by element, and land before the paths join.
  int n[R];
  Raw xr[R][E];
  Raw mr[R][E];               // AQSGD: the buffer row, kept for the update
  float er[R][E];             // EF: the residual
  // AQSGD: the example id, a scalar read, is waited for apart from the
  // input's loads
  int64_t id = 0;
  if constexpr (SEL == SEL_AQSGD) id = load_uniform(a.ids + seg);
  auto load_x = [&](auto vec_c) {
    constexpr bool VEC = decltype(vec_c)::value;
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const uint32_t off = (uint32_t)(j * NT + t) * E;
      n[j] = (int)min((uint32_t)E, (uint32_t)sat_sub(a.L, c0 + off));   // L < 2^32
      if constexpr (VEC) {
        load16_in<Raw, E, true>(xs, off, n[j] > 0, xr[j]);
      } else if (n[j] > 0) {
        load_run_partial<Raw, E, true>(xs + off, n[j], Raw{}, xr[j]);
      } else {
#pragma unroll
        for (int i = 0; i < E; ++i) xr[j][i] = Raw{};
      }
    }
    if constexpr (!VEC) __builtin_amdgcn_s_waitcnt(0);
  };
  if (vec) load_x(std::true_type{});
  else load_x(std::false_type{});
  Raw* ms = nullptr;
  if constexpr (SEL == SEL_AQSGD) {
    if (id < 0 || (uint64_t)id >= a.n_samples) {
      if (t == 0 && part == 0) raise_error(KERR_BAD_ID);
      return;                  // every workgroup of the group skips alike
    }
    ms = (Raw*)a.m + (uint64_t)id * a.L + c0;
  }
  auto load_me = [&](auto vec_c) {
    constexpr bool VEC = decltype(vec_c)::value;
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const uint32_t off = (uint32_t)(j * NT + t) * E;
      if constexpr (VEC) {
        const bool in = n[j] > 0;
        if constexpr (SEL == SEL_AQSGD) load16_in<Raw, E, true>(ms, off, in, mr[j]);
        if constexpr (SEL == SEL_EF) {
          if constexpr (E == 4) {
            load16_in<float, 4, true>(es, off, in, *reinterpret_cast<float(*)[4]>(&er[j][0]));
          } else {
            load16_in<float, 4, false>(es, off, in, *reinterpret_cast<float(*)[4]>(&er[j][0]));
            load16_in<float, 4, false>(es + 4, off, in, *reinterpret_cast<float(*)[4]>(&er[j][4]));
          }
        }
      } else if (n[j] > 0) {
        // elements past the segment's end read as +0 (x, m and e alike)
        if constexpr (SEL == SEL_AQSGD) load_run_partial<Raw, E, true>(ms + off, n[j], Raw{}, mr[j]);
        if constexpr (SEL == SEL_EF) load_run_partial<float, E, true>(es + off, n[j], 0.0f, er[j]);
      } else {
#pragma unroll
        for (int i = 0; i < E; ++i) { mr[j][i] = Raw{}; er[j][i] = 0.0f; }
      }
    }
    if constexpr (!VEC) __builtin_amdgcn_s_waitcnt(0);
  };
  if (vec) load_me(std::true_type{});
  else load_me(std::false_type{});
  // while the loads are in flight, exchange A's first histogram is cleared;
  // each run's keys go into it as soon as that run has landed
  const bool select = a.k != 0;
  if (select) grp_hist_clear<NT>(sh.sel, sm);
  float v[R][E];
  uint32_t zc = 0;
#pragma unroll
  for (int j = 0; j < R; ++j) {
#pragma unroll
    for (int i = 0; i < E; ++i) {
      float x = Elem<InT>::up(xr[j][i]);
      if constexpr (SEL == SEL_EF) x = x + er[j][i];
      if constexpr (SEL == SEL_AQSGD) x = x - Elem<InT>::up(mr[j][i]);
      v[j][i] = (n[j] > 0) ? x : 0.0f;     // +0 past the segment's end
    }
    if (select) {
#pragma unroll
      for (int i = 0; i < E; ++i) grp_hist_add(sh.sel, mag_key(v[j][i]), zc);
    }
  }
  // AQSGD: the buffer row waits in LDS for the update (it is not needed
  // before), which keeps it out of registers during the selection; a run
  // past the segment's end is never stored back
  if constexpr (SEL == SEL_AQSGD) {
#pragma unroll
    for (int j = 0; j < R; ++j) store16<Raw, E, false>(mlds + (uint32_t)(j * NT + t) * E, mr[j]);
  }

  // ---- selection (elements past the segment's end hold +0: see grp_exchange_a)
  // The early path (grp_early) needs registers of its own: with 16 or more
  // fp32 values (and their residuals) per thread it would spill, so those
  // layouts take the plain path.
  constexpr bool EARLY = !(sizeof(Raw) == 4 && R >= 4);
  SelResult sr;
  uint32_t ticket = 0;
  const bool exiting = P > 1 && last_seg;
  if (!select) {
    // T above every finite key (the keys of finite values are at most
    // 0x7F800000), so that nothing is kept
    sr.T = 0x7FFFFFFFu; sr.r = 0; sr.gt_before = 0; sr.eq_before = 0;
  } else {
    const SelA A = grp_exchange_a<NT, R, E, CH>(v, zc, (uint32_t)a.k, a.L, P, part, gm, sh.sel, sm, gs);
    refresh(v);
    bool cleared = false;
    if (EARLY && A.fine && P <= REC_P_MAX) {
      if (grp_early<InT, SEL, R>(a, vec, seg, P, part, gm, sh, sm, gs, A, v, n, c0, ms, es, mlds, exiting, ticket)) {
        if (exiting) {
          grp_exit_finish<NT>(gm, P, gs, ticket, &sm.misc[0]);
          exited = true;
        }
        __syncthreads();
        return;
      }
      cleared = true;
    }
    sr = grp_fallback<NT, R, E, CH>(v, P, part, gm, sh.sel, sm, gs, A.prefix, A.pbits, A.need, cleared);
  }
  // the group's exchange words have all been read: draw the exit ticket now
  // (its answer is needed only at the end)
  if (exiting) ticket = grp_exit_ticket(gm);

  refresh(v);
  // ---- placement: keys > T and == T per run, scanned over the workgroup
  // in index order (run-major, then thread); both counts stay below 2^16
  uint32_t pk[R], ex[R], tot[R];
#pragma unroll
  for (int j = 0; j < R; ++j) {
    uint32_t gt = 0, eq = 0;
#pragma unroll
    for (int i = 0; i < E; ++i) {
      // padding (+0 past the end) is never kept: it ranks after every element
      const uint32_t kk = mag_key(v[j][i]);
      gt += gt31(kk, sr.T);
      eq += eq31(kk, sr.T);
    }
    pk[j] = gt | (eq << 16);
  }
  block_excl_scan_multi<NT, R>(pk, ex, tot, sm.scratch);
  uint32_t eq_wg = 0;
#pragma unroll
  for (int j = 0; j < R; ++j) eq_wg += tot[j] >> 16;
  const uint32_t quota_wg = min(sat_sub(sr.r, sr.eq_before), eq_wg);   // ties this workgroup keeps
  const uint32_t wg_first = sr.gt_before + min(sr.eq_before, sr.r);
  uint32_t pos0[R], tie_keep[R], kept_before[R];
  uint32_t eq_run = 0, kept_run = 0;
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const uint32_t gtt = tot[j] & 0xFFFFu, eqt = tot[j] >> 16;
    const uint32_t gx = ex[j] & 0xFFFFu, qx = ex[j] >> 16;
    const uint32_t quota_j = min(sat_sub(quota_wg, eq_run), eqt);    // ties kept in run j
    kept_before[j] = kept_run;
    pos0[j] = kept_run + gx + min(qx, quota_j);
    tie_keep[j] = min(pk[j] >> 16, sat_sub(quota_j, qx));
    eq_run += eqt;
    kept_run += gtt + quota_j;
  }
  const uint32_t wg_count = kept_run;

  refresh(v);
  // ---- payload into LDS + epilogue (entries not kept write to the lane's
  // dummy slot)
  uint32_t overflow = 0;
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const uint32_t off = (uint32_t)(j * NT + t) * E;
    uint32_t pos = pos0[j], ties = 0;
    float eo[E];
    if constexpr (SEL == SEL_AQSGD) load16<Raw, E, false>(mlds + off, mr[j]);
#pragma unroll
    for (int i = 0; i < E; ++i) {
      const uint32_t kk = mag_key(v[j][i]);
      const uint32_t tie = eq31(kk, sr.T);
      const uint32_t kept = gt31(kk, sr.T) | (tie & gt31(tie_keep[j], ties));
      ties += tie;
      const Raw w = Elem<InT>::down(v[j][i]);
      const uint32_t fits = gt31(CH, pos);               // pos < CH (never false when kept)
      overflow |= kept & (fits ^ 1u);
      const uint32_t slot = pick(kept & fits, pos, CH + dummy);
      sh.st.idx[slot] = (uint32_t)c0 + off + (uint32_t)i;
      sh.st.val[slot] = w;
      pos += kept;
      if constexpr (SEL == SEL_AQSGD) {
        const Raw upd = Elem<InT>::down(Elem<InT>::up(mr[j][i]) + Elem<InT>::up(w));
        if constexpr (sizeof(Raw) == 4) mr[j][i] = __uint_as_float(pick(kept, __float_as_uint(upd), __float_as_uint(mr[j][i])));
        else mr[j][i] = (Raw)pick(kept, upd, mr[j][i]);
      }
      if constexpr (SEL == SEL_EF) eo[i] = v[j][i] - __uint_as_float(pick(kept, __float_as_uint(through<InT>(v[j][i])), 0u));
    }
    // a run of 16 bytes per lane is one store instruction covering 1 KiB
    // (non-temporal: whole lines); an fp32 residual of 8 elements is two per
    // lane, which write-back stores let the L2 merge
    if (vec && n[j] == E) {
      if constexpr (SEL == SEL_EF) {
        if constexpr (E == 4) {
          store16<float, 4, true>(es + off, *reinterpret_cast<float(*)[4]>(&eo[0]));
        } else {
          store16<float, 4, false>(es + off, *reinterpret_cast<float(*)[4]>(&eo[0]));
          store16<float, 4, false>(es + off + 4, *reinterpret_cast<float(*)[4]>(&eo[4]));
        }
      }
      if constexpr (SEL == SEL_AQSGD) store16<Raw, E, true>(ms + off, mr[j]);
    } else if (n[j] > 0) {
      if constexpr (SEL == SEL_EF) store_run_partial<float, E, true>(es + off, n[j], eo);
      if constexpr (SEL == SEL_AQSGD) store_run_partial<Raw, E, true>(ms + off, n[j], mr[j]);
    }
  }
  if (overflow) raise_error(KERR_INTERNAL);
  __syncthreads();
  // the workgroup's run of the payload, in index order, coalesced
  uint32_t* idx = a.idx + seg * a.k;
  Raw* val = (Raw*)a.val + seg * a.k;
  const uint32_t cnt = min(wg_count, CH);
  if (wg_first + cnt > a.k) {
    if (t == 0) raise_error(KERR_INTERNAL);
  } else {
    copy_lds_to_global<NT>(idx + wg_first, sh.st.idx, cnt);
    copy_lds_to_global<NT>(val + wg_first, sh.st.val, cnt);
  }
  // block table: kept entries below each block boundary this workgroup
  // covers.  Block boundaries are multiples of 4096 elements and runs span
  // NT*E (4096 or 2048) elements, so each boundary starts a run: the count
  // is the workgroup's first slot plus the runs before it.
  static_assert(BLOCK_LEN % ((uint64_t)NT * E) == 0 && CH % ((uint64_t)NT * E) == 0, "block boundaries start runs");
  if (a.blk && t == 0) {
    uint32_t* bt = a.blk + seg * (n_blocks(a.L) + 1);
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const uint64_t B = c0 + (uint64_t)j * NT * E;
      if (B % BLOCK_LEN == 0 && B < a.L) bt[B / BLOCK_LEN] = wg_first + kept_before[j];
    }
    if (part == 0) bt[n_blocks(a.L)] = (uint32_t)a.k;
  }
  if (exiting) {
    grp_exit_finish<NT>(gm, P, gs, ticket, &sm.misc[0]);
    exited = true;
  }
  __syncthreads();
}

template <typename InT, int SEL, int R>
__global__ __launch_bounds__(GRP_NT) void k_topk_grp(TopkArgs a) {
  using Raw = typename Elem<InT>::raw;
  constexpr int E = 16 / (int)sizeof(Raw);            // elements per 16-byte run
  constexpr uint32_t CH = (uint32_t)GRP_NT * R * E;    // elements per workgroup
  __shared__ GrpShared<CH, Raw> sh;
  __shared__ GrpSmall sm;
  __shared__ __attribute__((aligned(16))) Raw mlds[SEL == SEL_AQSGD ? CH : 8];   // the buffer row (AQSGD)

  const uint32_t P = a.P;
  uint32_t group, part;
  map_wg(blockIdx.x, gridDim.x, P, group, part);
  const uint32_t n_groups = gridDim.x / P;
  GrpMem gm{};
  if (P > 1) gm = grp_mem(a.ws, group, P);
  GrpState gs;
  bool exited = false;
  // whole 16-byte runs everywhere: every buffer 16-byte aligned, segment
  // starts too (L a multiple of the run length), and this chunk inside the segment
  const uintptr_t al = (uintptr_t)a.x | (uintptr_t)a.e | (uintptr_t)a.m;
  const bool vec = (al & 15u) == 0 && (a.L % E) == 0;

  if (a.n_seg <= n_groups) {
    // one segment per group (a straight path: nothing for the compiler to
    // hoist out of a loop and keep in registers)
    if (group < a.n_seg) grp_segment<InT, SEL, R>(a, vec, group, P, part, gm, sh, sm, gs, true, exited, mlds);
  } else {
    for (uint64_t seg = group; seg < a.n_seg; seg += n_groups, ++gs.iter) {
      const bool last_seg = seg + n_groups >= a.n_seg;
      grp_segment<InT, SEL, R>(a, vec, seg, P, part, gm, sh, sm, gs, last_seg, exited, mlds);
    }
  }
  if (P > 1 && !exited) {
    const uint32_t ticket = grp_exit_ticket(gm);
    grp_exit_finish<GRP_NT>(gm, P, gs, ticket, &sm.misc[0]);
  }
}

// ------------------------------------------------------------- LDS engine
// One workgroup per segment of up to LDS_MAX elements (per-sample CNN
// activations and gradients, short AQ-SGD / EF21 rows): the segment's values
// v = x (+ e), or a - m, stay in LDS as binary32 for the whole selection, so
// no other workgroup takes part and nothing crosses the workgroup.  Loads are
// lane-consecutive 4-element pieces; three digit passes over LDS (key bits
// 30..19, 18..7, 6..0) give T and the tie quota; then thread t places its run
// of LDS_RUN consecutive elements (kept-entry bit masks, one scan), writes
// its kept entries to the payload and its residual (EF) or moves the buffer
// row at its kept entries (AQ-SGD).  1024 threads: four waves per SIMD share
// the per-key work, which is what bounds this kernel.
constexpr int LDS_NT = 1024;
constexpr uint32_t LDS_MAX = 32768;
constexpr uint32_t LDS_RUN = LDS_MAX / LDS_NT;   // 32: one bit mask word per thread
constexpr uint32_t LDS_PIECES = LDS_RUN / 4;     // 4-element pieces per thread
constexpr uint32_t LDS_LIST = 3072;              // keys of one first-pass bin kept in a list
static_assert(LDS_RUN == 32, "a thread's run is one 32-bit mask");
static_assert(BLOCK_LEN % LDS_RUN == 0, "block boundaries start a thread's run");

// One digit pass: counts of bits [shift, shift + width) of the keys whose
// bits above them equal `prefix` (shift + width = 31: every key); the digit
// holding the need-th largest such key goes to `digit`, need becomes its
// rank inside that digit.  Exact zeros (their digits are all 0) are counted
// in registers and added once per wavefront, off one hot bin.  A piece of
// four keys none of which matches costs one test.
template <int NT, int NB>
__device__ __forceinline__ void lds_pass(const uint32_t* s_v, uint32_t L, uint32_t shift, uint32_t prefix,
                                         uint32_t* s_h, uint32_t* scratch, uint32_t* found, uint32_t& need,
                                         uint32_t& digit) {
  static_assert(NB == 4096 || NB == LAST_BINS, "12-bit or 7-bit digits");
  constexpr uint32_t width = (NB == 4096) ? 12u : 7u;
  const uint32_t t = threadIdx.x;
  for (uint32_t b = t; b < (uint32_t)NB; b += NT) s_h[b] = 0u;
  __syncthreads();
  uint32_t zc = 0;
  for (uint32_t q = t; q * 4 < L; q += NT) {
    const u32x4 w = *reinterpret_cast<const u32x4*>(&s_v[q * 4]);
    uint32_t kk[4], in = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      kk[c] = w[c] & 0x7FFFFFFFu;
      in |= (((kk[c] >> (shift + width)) == prefix) ? 1u : 0u) << c;
    }
    if (q * 4 + 4 > L) in &= (1u << (L - q * 4)) - 1u;
    if (in) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if ((in >> c) & 1u) {
          if (kk[c] == 0u) ++zc;
          else atomicAdd(&s_h[(kk[c] >> shift) & (uint32_t)(NB - 1)], 1u);
        }
      }
    }
  }
  const uint32_t zs = wave_sum(zc);
  if (lane_id() == 0 && zs) atomicAdd(&s_h[0], zs);
  __syncthreads();
  if constexpr (NB == 4096) find_bin<NT, NB>(s_h, need, scratch, found);
  else find_bin_wave<NB>(s_h, need, found);
  digit = found[0];
  need -= found[1];
  __syncthreads();
}

// The same over the short list of keys of one first-pass bin: bits
// [shift, shift + width) of the listed keys (all of them for the 12-bit
// digit; for the 7-bit digit those whose bits 30..7 equal `prefix`).
template <int NT, int NB>
__device__ __forceinline__ void lds_pass_list(const uint32_t* s_list, uint32_t n, uint32_t shift, uint32_t* s_h,
                                              uint32_t* scratch, uint32_t* found, uint32_t& need, uint32_t& digit,
                                              uint32_t prefix = 0u) {
  const uint32_t t = threadIdx.x;
  for (uint32_t b = t; b < (uint32_t)NB; b += NT) s_h[b] = 0u;
  __syncthreads();
  for (uint32_t j = t; j < n; j += NT) {
    const uint32_t kk = s_list[j];
    if (NB == 4096 || (kk >> 7) == prefix) atomicAdd(&s_h[(kk >> shift) & (uint32_t)(NB - 1)], 1u);
  }
  __syncthreads();
  if constexpr (NB == 4096) find_bin<NT, NB>(s_h, need, scratch, found);
  else find_bin_wave<NB>(s_h, need, found);
  digit = found[0];
  need -= found[1];
  __syncthreads();
}

// T (the key of the k-th largest |v| in s_v[0..L)) and the tie quota r:
// the number of keys equal to T that are kept (k == 0: T above every
// finite key).  Ends with every thread past a barrier.  LIST: the keys of
// the first digit's bin go to a short list for the last two passes (else
// those passes read the whole segment).
// hist_ready: s_h already holds the first digit's counts of every key (the
// load loop counted them as the values arrived); only the search is left.
template <int NT, bool LIST = true>
__device__ __forceinline__ void lds_threshold(const uint32_t* s_v, uint32_t L, uint32_t k, uint32_t* s_h,
                                              uint32_t* s_list, uint32_t* scratch, uint32_t* found, uint32_t& T,
                                              uint32_t& r, bool hist_ready = false) {
  const uint32_t t = threadIdx.x;
  T = 0x7FFFFFFFu;
  r = 0u;
  if (k > 0) {
    uint32_t need = k, d1, d2, d3;
    if (hist_ready) {
      find_bin<NT, 4096>(s_h, need, scratch, found);
      d1 = found[0];
      need -= found[1];
      __syncthreads();
    } else {
      lds_pass<NT, 4096>(s_v, L, 19, 0u, s_h, scratch, found, need, d1);
    }
    uint32_t nl = LDS_LIST + 1u;
    if constexpr (LIST) {
      // the keys of bin d1 into a short list, so that the last two passes
      // read only them (a bin holding more than the list takes the passes
      // over the whole segment): each thread marks its matches in one mask
      // (bit 4j + c: element c of its piece j), one wavefront scan and one
      // append per wavefront place them, and the few matches are read again
      if (t == 0) found[0] = 0u;
      __syncthreads();
      uint32_t mask = 0;
#pragma unroll
      for (uint32_t j = 0; j < LDS_PIECES; ++j) {
        const uint32_t q = j * NT + t;
        if (q * 4 >= L) continue;
        const u32x4 w = *reinterpret_cast<const u32x4*>(&s_v[q * 4]);
        uint32_t in = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c) in |= ((((w[c] & 0x7FFFFFFFu) >> 19) == d1) ? 1u : 0u) << c;
        if (q * 4 + 4 > L) in &= (1u << (L - q * 4)) - 1u;
        mask |= in << (4 * j);
      }
      const uint32_t n = (uint32_t)__builtin_popcount(mask);
      const uint32_t incl = wave_incl_scan(n);
      const uint32_t tot_w = (uint32_t)__builtin_amdgcn_readlane((int)incl, WAVE - 1);
      uint32_t base = 0;
      if (tot_w) {
        if (lane_id() == 0) base = atomicAdd(&found[0], tot_w);
        base = (uint32_t)__builtin_amdgcn_readfirstlane((int)base);
      }
      uint32_t o = base + incl - n;
      for (uint32_t m = mask; m; m &= m - 1u) {
        const uint32_t bit = (uint32_t)__builtin_ctz(m);
        const uint32_t i = ((bit >> 2) * NT + t) * 4 + (bit & 3u);
        if (o < LDS_LIST) s_list[o] = s_v[i] & 0x7FFFFFFFu;
        ++o;
      }
      __syncthreads();
      nl = found[0];
      __syncthreads();
    }
    if (nl <= LDS_LIST) {
      lds_pass_list<NT, 4096>(s_list, nl, 7, s_h, scratch, found, need, d2);
      lds_pass_list<NT, LAST_BINS>(s_list, nl, 0, s_h, scratch, found, need, d3, (d1 << 12) | d2);
    } else {
      lds_pass<NT, 4096>(s_v, L, 7, d1, s_h, scratch, found, need, d2);
      lds_pass<NT, LAST_BINS>(s_v, L, 0, (d1 << 12) | d2, s_h, scratch, found, need, d3);
    }
    T = (d1 << 19) | (d2 << 7) | d3;
    r = need;
  }
}

// Placement: thread t owns the run [b0, b0 + nr) of LDS_RUN consecutive
// elements; its pieces are read in an order rotated by t (fewer LDS bank
// conflicts) and flags go to bit (element - b0) of two masks.  The kept
// entries go to idx / val (in index order) and the block table (or null);
// returns the thread's kept-entry mask.
template <typename InT, int NT>
__device__ __forceinline__ uint32_t lds_place(const uint32_t* s_v, uint32_t L, uint32_t b0, uint32_t nr, uint32_t T,
                                              uint32_t r, uint32_t k, uint32_t* idx, typename Elem<InT>::raw* val,
                                              uint32_t* bt, uint32_t* scratch) {
  const uint32_t t = threadIdx.x;
  uint32_t gm = 0, em = 0;
#pragma unroll
  for (uint32_t j = 0; j < LDS_PIECES; ++j) {
    const uint32_t pc = (j + t) % LDS_PIECES;
    const u32x4 w = *reinterpret_cast<const u32x4*>(&s_v[b0 + 4 * pc]);
    uint32_t g4 = 0, e4 = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const uint32_t kk = w[c] & 0x7FFFFFFFu;
      g4 |= ((kk > T) ? 1u : 0u) << c;
      e4 |= ((kk == T) ? 1u : 0u) << c;
    }
    gm |= g4 << (4 * pc);
    em |= e4 << (4 * pc);
  }
  const uint32_t valid = (nr >= 32u) ? 0xFFFFFFFFu : ((1u << nr) - 1u);
  gm &= valid;
  em &= valid;
  const uint32_t gt = (uint32_t)__builtin_popcount(gm), eq = (uint32_t)__builtin_popcount(em);
  uint32_t tot;
  const uint32_t ex = block_excl_scan<NT>(gt | (eq << 16), scratch, tot);   // both < 2^16
  const uint32_t gt_ex = ex & 0xFFFFu, eq_ex = ex >> 16;
  // ties kept: the r lowest-indexed ones
  uint32_t tie_keep = min(sat_sub(r, eq_ex), eq);
  uint32_t km = gm, rest = em;
  for (; tie_keep; --tie_keep) {
    km |= rest & (0u - rest);
    rest &= rest - 1u;
  }
  const uint32_t pos0 = gt_ex + min(eq_ex, r);
  const uint32_t nk = (uint32_t)__builtin_popcount(km);
  if (pos0 + nk > k) {
    raise_error(KERR_INTERNAL);
    km = 0;
  }
  // the kept entries, in index order
  uint32_t pos = pos0;
  for (uint32_t m = km; m; m &= m - 1u) {
    const uint32_t bit = (uint32_t)__builtin_ctz(m);
    idx[pos] = b0 + bit;
    val[pos] = Elem<InT>::down(__uint_as_float(s_v[b0 + bit]));
    ++pos;
  }
  // block table: kept entries below each block boundary (a boundary
  // starts a thread's run)
  if (bt) {
    if (b0 % BLOCK_LEN == 0 && b0 < L) bt[b0 / BLOCK_LEN] = pos0;
    if (t == 0) bt[n_blocks(L)] = k;
  }
  return km;
}

template <typename InT, int SEL>
__global__ __launch_bounds__(LDS_NT) void k_topk_lds(TopkArgs a) {
  using Raw = typename Elem<InT>::raw;
  constexpr int NT = LDS_NT;
  __shared__ __attribute__((aligned(16))) uint32_t s_v[LDS_MAX];   // the segment's values (binary32 bits)
  __shared__ uint32_t s_h[HIST_BINS + WAVE];   // histograms (the last WAVE words: per-lane dummies)
  __shared__ uint32_t s_list[LDS_LIST];   // keys of the first pass's bin
  __shared__ uint32_t scratch[NT / WAVE + 2];
  __shared__ uint32_t found[2];
  const uint32_t t = threadIdx.x;
  const uint32_t L = (uint32_t)a.L;   // <= LDS_MAX (the plan guarantees it)
  const bool vec = ((((uintptr_t)a.x | (uintptr_t)a.e | (uintptr_t)a.m) & 15u) == 0) && (L % 4u) == 0;
  // EF-mixed: two work items per segment, the input's selection (even) and
  // the buffer's (odd), independent of each other; the residual follows in
  // a kernel of its own
  const uint64_t n_items = (SEL == SEL_EFMIX) ? 2 * a.n_seg : a.n_seg;
  for (uint64_t item = blockIdx.x; item < n_items; item += gridDim.x) {
    const uint64_t seg = (SEL == SEL_EFMIX) ? item >> 1 : item;
    const bool buf_list = (SEL == SEL_EFMIX) && (item & 1u);
    const Raw* xs = (const Raw*)a.x + seg * a.L;
    float* es = (SEL == SEL_EF || SEL == SEL_EFMIX) ? a.e + seg * a.L : nullptr;
    // AQ-SGD: the example's buffer row; v = a - m
    Raw* ms = nullptr;
    if constexpr (SEL == SEL_AQSGD) {
      const int64_t id = load_uniform(a.ids + seg);
      if (id < 0 || (uint64_t)id >= a.n_samples) {
        if (t == 0) raise_error(KERR_BAD_ID);
        continue;                  // every thread skips alike
      }
      ms = (Raw*)a.m + (uint64_t)id * a.L;
    }
    // ---- values into LDS: piece q = 4 elements, lanes consecutive; loads
    // go out four pieces at a time (the registers of 1024 threads).  The
    // first digit pass (key bits 30..19) is counted here, from registers, as
    // the values arrive; exact zeros are counted apart and added once per
    // wavefront (padding past the segment's end is not counted)
    for (uint32_t b = t; b < (uint32_t)HIST_BINS; b += NT) s_h[b] = 0u;
    __syncthreads();
    const uint32_t dummy = HIST_BINS + (uint32_t)lane_id();
    uint32_t zc = 0;
    auto count = [&](uint32_t bits) {
      const uint32_t kk = bits & 0x7FFFFFFFu;
      const uint32_t z = eq31(kk, 0u);
      zc += z;
      atomicAdd(&s_h[pick(z, dummy, kk >> 19)], 1u);
    };
    if constexpr (SEL == SEL_EFMIX) {
      // one array per workgroup, x or the buffer e, the source and the
      // alignment case chosen once (a choice per piece would put each load
      // in a branch of its own and serialise them); cached loads, as the
      // residual kernel reads both again
      auto fill = [&](auto from_e, auto vec_c) {
        constexpr bool FE = decltype(from_e)::value;
        constexpr bool VEC = decltype(vec_c)::value;
#pragma unroll
        for (uint32_t h = 0; h < LDS_PIECES; h += 4) {
          float f[4][4];
#pragma unroll
          for (uint32_t j = 0; j < 4; ++j) {
            const uint32_t i0 = ((h + j) * NT + t) * 4;
            if constexpr (VEC) {
              // a piece past the segment's end reads the first piece
              // (unused), so that no branch stands between the loads
              const uint32_t ia = (i0 < L) ? i0 : 0u;
              if constexpr (FE) {
                load16<float, 4, false>(es + ia, f[j]);
              } else if constexpr (sizeof(Raw) == 4) {
                load16<float, 4, false>(reinterpret_cast<const float*>(xs) + ia, f[j]);
              } else {
                Raw xr[4];
                load_piece<Raw, false>(xs + ia, xr);
#pragma unroll
                for (int c = 0; c < 4; ++c) f[j][c] = Elem<InT>::up(xr[c]);
              }
            } else {
#pragma unroll
              for (int c = 0; c < 4; ++c) {
                const uint32_t i = i0 + (uint32_t)c;
                if constexpr (FE) f[j][c] = (i < L) ? es[i] : 0.0f;
                else f[j][c] = (i < L) ? Elem<InT>::up(xs[i]) : 0.0f;
              }
            }
          }
#pragma unroll
          for (uint32_t j = 0; j < 4; ++j) {
            const uint32_t i0 = ((h + j) * NT + t) * 4;
            if (i0 < L) {
              u32x4 w;
#pragma unroll
              for (int c = 0; c < 4; ++c) {
                w[c] = __float_as_uint(f[j][c]);
                if (i0 + (uint32_t)c < L) count(w[c]);
              }
              *reinterpret_cast<u32x4*>(&s_v[i0]) = w;
            }
          }
        }
      };
      if (buf_list) {
        if (vec) fill(std::true_type{}, std::true_type{});
        else fill(std::true_type{}, std::false_type{});
      } else {
        if (vec) fill(std::false_type{}, std::true_type{});
        else fill(std::false_type{}, std::false_type{});
      }
    } else if (vec) {
#pragma unroll
      for (uint32_t h = 0; h < LDS_PIECES; h += 4) {
        Raw xr[4][4], mr[4][4];
        float er[4][4];
#pragma unroll
        for (uint32_t j = 0; j < 4; ++j) {
          // (vec: pieces aligned and whole; one past the segment's end
          // reads the first piece, unused, so that no branch stands between
          // the loads)
          const uint32_t i0 = ((h + j) * NT + t) * 4;
          const uint32_t ia = (i0 < L) ? i0 : 0u;
          load_piece<Raw, true>(xs + ia, xr[j]);
          if constexpr (SEL == SEL_EF) load_piece<float, true>(es + ia, er[j]);
          if constexpr (SEL == SEL_AQSGD) load_piece<Raw, true>(ms + ia, mr[j]);
        }
#pragma unroll
        for (uint32_t j = 0; j < 4; ++j) {
          const uint32_t i0 = ((h + j) * NT + t) * 4;
          if (i0 < L) {
            u32x4 w;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
              float x = Elem<InT>::up(xr[j][c]);
              if constexpr (SEL == SEL_EF) x = x + er[j][c];
              if constexpr (SEL == SEL_AQSGD) x = x - Elem<InT>::up(mr[j][c]);
              w[c] = __float_as_uint(x);
              count(w[c]);
            }
            *reinterpret_cast<u32x4*>(&s_v[i0]) = w;
          }
        }
      }
    } else {
      for (uint32_t j = 0; j < LDS_PIECES; ++j) {
        const uint32_t i0 = (j * NT + t) * 4;
        if (i0 >= L) break;
        u32x4 w;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const uint32_t i = i0 + (uint32_t)c;
          float x = 0.0f;
          if (i < L) {
            x = Elem<InT>::up(xs[i]);
            if constexpr (SEL == SEL_EF) x = x + es[i];
            if constexpr (SEL == SEL_AQSGD) x = x - Elem<InT>::up(ms[i]);
            count(__float_as_uint(x));
          }
          w[c] = __float_as_uint(x);
        }
        *reinterpret_cast<u32x4*>(&s_v[i0]) = w;
      }
    }
    {
      const uint32_t zs = wave_sum(zc);
      if (lane_id() == 0 && zs) atomicAdd(&s_h[0], zs);
    }
    __syncthreads();

    // ---- T and the tie quota r, then the kept entries of thread t's run
    uint32_t T, r;
    const uint64_t kk = buf_list ? a.k2 : a.k;
    uint32_t* const lidx = buf_list ? a.idx2 : a.idx;
    Raw* const lval = (Raw*)(buf_list ? a.val2 : a.val);
    uint32_t* const lblk = buf_list ? a.blk2 : a.blk;
    lds_threshold<NT, true>(s_v, L, (uint32_t)kk, s_h, s_list, scratch, found, T, r, true);
    const uint32_t b0 = t * LDS_RUN;
    const uint32_t nr = (b0 < L) ? min(LDS_RUN, L - b0) : 0u;
    const uint32_t km = lds_place<InT, NT>(s_v, L, b0, nr, T, r, (uint32_t)kk, lidx + seg * kk, lval + seg * kk,
                                           lblk ? lblk + seg * (n_blocks(a.L) + 1) : nullptr, scratch);
    // AQ-SGD: the buffer row moves by the sent values at the kept entries
    // only; per half of the run, that half's buffer values are loaded at once
    if constexpr (SEL == SEL_AQSGD) {
#pragma unroll
      for (uint32_t hh = 0; hh < LDS_RUN; hh += 16) {
        const uint32_t kh = (km >> hh) & 0xFFFFu;
        if (kh == 0u) continue;
        Raw mo[16];
        if (vec && hh + 16 <= nr) {
          load_run<Raw, 16, false>(ms + b0 + hh, mo);
        } else {
#pragma unroll
          for (uint32_t c = 0; c < 16; ++c) mo[c] = (hh + c < nr) ? ms[b0 + hh + c] : Raw{};
        }
#pragma unroll
        for (uint32_t c = 0; c < 16; ++c) {
          if ((kh >> c) & 1u) {
            const Raw w = Elem<InT>::down(__uint_as_float(s_v[b0 + hh + c]));
            ms[b0 + hh + c] = Elem<InT>::down(Elem<InT>::up(mo[c]) + Elem<InT>::up(w));
          }
        }
      }
    }
    // the residual: v minus what the receiver holds, in the load's layout
    // (lanes consecutive: whole lines per wavefront store); the kept masks
    // of the runs go through LDS
    if constexpr (SEL == SEL_EF) {
      s_h[t] = km;
      uint32_t tq = t;
      asm volatile("" : "+v"(tq));   // addresses computed here, not ahead of the loop
      __syncthreads();
#pragma unroll
      for (uint32_t j = 0; j < LDS_PIECES; ++j) {
        const uint32_t i0 = (j * NT + tq) * 4;
        if (i0 >= L) continue;
        const u32x4 w = *reinterpret_cast<const u32x4*>(&s_v[i0]);
        const uint32_t k4 = s_h[i0 / LDS_RUN] >> (i0 % LDS_RUN);
        float o[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const float v = __uint_as_float(w[c]);
          o[c] = v - (((k4 >> c) & 1u) ? through<InT>(v) : 0.0f);
        }
        if (vec) store_run<float, 4, true>(es + i0, o);
        else {
#pragma unroll
          for (int c = 0; c < 4; ++c)
            if (i0 + (uint32_t)c < L) es[i0 + c] = o[c];
        }
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ plans
namespace {

constexpr uint64_t ROW_MAX = (uint64_t)WAVE * 32;   // longest segment one wavefront holds
static_assert(ROW_MAX <= BLOCK_LEN, "a wavefront segment fits in one block of the block table");

template <typename InT, int SEL>
const void* row_ptr(int vpt) {
  switch (vpt) {
    case 4: return (const void*)k_topk_row<InT, SEL, 4>;
    case 8: return (const void*)k_topk_row<InT, SEL, 8>;
    case 12: return (const void*)k_topk_row<InT, SEL, 12>;
    case 16: return (const void*)k_topk_row<InT, SEL, 16>;
    case 24: return (const void*)k_topk_row<InT, SEL, 24>;
    case 32: return (const void*)k_topk_row<InT, SEL, 32>;
  }
  return nullptr;
}

// group engine: R runs of 16 bytes per thread (VPT = R * elements per run)
template <typename InT, int SEL>
const void* grp_ptr(int r) {
  if constexpr (sizeof(typename Elem<InT>::raw) == 4) {
    switch (r) {
      case 1: return (const void*)k_topk_grp<InT, SEL, 1>;
      case 2: return (const void*)k_topk_grp<InT, SEL, 2>;
      case 4: return (const void*)k_topk_grp<InT, SEL, 4>;
      case 6: return (const void*)k_topk_grp<InT, SEL, 6>;
    }
  } else {
    switch (r) {
      case 1: return (const void*)k_topk_grp<InT, SEL, 1>;
      case 2: return (const void*)k_topk_grp<InT, SEL, 2>;
      case 3: return (const void*)k_topk_grp<InT, SEL, 3>;
    }
  }
  return nullptr;
}

template <int SEL>
const void* pick_sel(int dt, bool row, int v) {
  if (dt == DT_F32) return row ? row_ptr<float, SEL>(v) : grp_ptr<float, SEL>(v);
  if (dt == DT_BF16) return row ? row_ptr<bf16_t, SEL>(v) : grp_ptr<bf16_t, SEL>(v);
  return row ? row_ptr<f16_t, SEL>(v) : grp_ptr<f16_t, SEL>(v);
}

// v: the row engine's elements per thread, or the group engine's runs per thread
const void* pick(int sel, int dt, bool row, int v) {
  if (sel == SEL_PLAIN) return pick_sel<SEL_PLAIN>(dt, row, v);
  if (sel == SEL_EF) return pick_sel<SEL_EF>(dt, row, v);
  return pick_sel<SEL_AQSGD>(dt, row, v);
}

// LDS engine: plain, EF, AQ-SGD and EF-mixed TopK
const void* lds_ptr(int sel, int dt) {
  if (sel == SEL_PLAIN) {
    if (dt == DT_F32) return (const void*)k_topk_lds<float, SEL_PLAIN>;
    if (dt == DT_BF16) return (const void*)k_topk_lds<bf16_t, SEL_PLAIN>;
    return (const void*)k_topk_lds<f16_t, SEL_PLAIN>;
  }
  if (sel == SEL_EF) {
    if (dt == DT_F32) return (const void*)k_topk_lds<float, SEL_EF>;
    if (dt == DT_BF16) return (const void*)k_topk_lds<bf16_t, SEL_EF>;
    return (const void*)k_topk_lds<f16_t, SEL_EF>;
  }
  if (sel == SEL_EFMIX) {
    if (dt == DT_F32) return (const void*)k_topk_lds<float, SEL_EFMIX>;
    if (dt == DT_BF16) return (const void*)k_topk_lds<bf16_t, SEL_EFMIX>;
    return (const void*)k_topk_lds<f16_t, SEL_EFMIX>;
  }
  if (dt == DT_F32) return (const void*)k_topk_lds<float, SEL_AQSGD>;
  if (dt == DT_BF16) return (const void*)k_topk_lds<bf16_t, SEL_AQSGD>;
  return (const void*)k_topk_lds<f16_t, SEL_AQSGD>;
}

int occupancy(const void* fn, int nt) {
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, fn, nt, 0) != hipSuccess || blocks < 1) blocks = 1;
  return blocks;
}

}  // namespace

static_assert(LDS_MAX == LDS_SEG_MAX, "one LDS-engine segment length");

// one workgroup per segment, the segment in LDS
SegPlan plan_lds(int sel, int dt, uint64_t n_seg) {
  SegPlan p;
  p.nt = LDS_NT;
  p.lds = true;
  p.P = 1;
  const uint64_t cap = (uint64_t)occupancy(lds_ptr(sel, dt), p.nt) * (uint32_t)device_cus();
  p.capacity = cap;
  p.n_groups = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(n_seg, cap));
  p.grid = p.n_groups;
  p.ws_words = 0;
  return p;
}

SegPlan plan_topk(int sel, int dt, uint64_t n_seg, uint64_t L) {
  SegPlan p;
  const uint32_t cus = (uint32_t)device_cus();
  if (L > ROW_MAX && L <= LDS_MAX) return plan_lds(sel, dt, n_seg);
  if (L <= ROW_MAX) {
    // one wavefront per segment: the smallest run length that covers L
    static const int vpts[] = {4, 8, 12, 16, 24, 32};
    p.nt = WAVE;
    for (int v : vpts) { p.vpt = v; if ((uint64_t)WAVE * v >= L) break; }
    p.P = 1;
    const uint64_t cap = (uint64_t)occupancy(pick(sel, dt, true, p.vpt), p.nt) * cus;
    p.capacity = cap;
    p.n_groups = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(n_seg, cap));
    p.grid = p.n_groups;
    p.ws_words = 0;
    return p;
  }
  // several workgroups per segment: the most 16-byte runs per thread that
  // still give every compute unit a workgroup, else the fewest
  const int E = (dt == DT_F32) ? 4 : 8;
  static const int runs32[] = {6, 4, 2, 1};
  static const int runs16[] = {3, 2, 1};
  const int* runs = (dt == DT_F32) ? runs32 : runs16;
  const int n_runs = (dt == DT_F32) ? 4 : 3;
  p.nt = GRP_NT;
  p.vpt = runs[n_runs - 1];   // runs per thread
  for (int i = 0; i < n_runs; ++i) {
    const uint64_t ch = (uint64_t)GRP_NT * runs[i] * E;
    const uint64_t P = (L + ch - 1) / ch;
    if (n_seg * P >= cus) { p.vpt = runs[i]; break; }
  }
  const uint64_t CH = (uint64_t)GRP_NT * p.vpt * E;
  const uint64_t P = (L + CH - 1) / CH;
  const uint64_t cap = (uint64_t)occupancy(pick(sel, dt, false, p.vpt), p.nt) * cus;
  p.capacity = cap;
  if (P > GRP_MAX_P) {       // too long for one resident group: the caller takes the global chain
    p.P = (uint32_t)std::min<uint64_t>(P, UINT32_MAX);
    p.n_groups = 0;
    return p;
  }
  p.P = (uint32_t)P;
  uint64_t groups = std::min<uint64_t>(n_seg, std::max<uint64_t>(1, cap / p.P));
  if (p.P > 1 && groups >= 8) groups -= groups % 8;
  p.n_groups = (uint32_t)groups;
  p.grid = (uint32_t)(groups * p.P);
  // the workspace is sized for the most groups any instance could keep
  // resident (4 workgroups per compute unit), so that one size serves every
  // selection kind of the same layout
  const uint64_t ws_groups = std::min<uint64_t>(n_seg, std::max<uint64_t>(1, (uint64_t)cus * 4 / p.P));
  p.ws_words = (p.P > 1) ? ws_groups * grp_mem_words(p.P) : 0;
  p.ws_used = (p.P > 1) ? groups * grp_mem_words(p.P) : 0;
  return p;
}

hipError_t launch_topk(int sel, int dt, const SegPlan& plan, const TopkArgs& args, hipStream_t st) {
  const void* fn = plan.lds ? lds_ptr(sel, dt) : pick(sel, dt, plan.nt == WAVE, plan.vpt);
  if (!fn) return hipErrorInvalidValue;
  TopkArgs a = args;
  a.P = plan.P;
  void* params[] = {&a};
  return hipLaunchKernel(fn, dim3(plan.grid), dim3(plan.nt), params, 0, st);
}

TC_DEFINE_ERROR_READER(errors_topk)

}  // namespace tc
