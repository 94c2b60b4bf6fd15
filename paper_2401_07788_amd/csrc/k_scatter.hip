// k_scatter.hip -- the receiver side of TopK (Sec. 2.3: the dense tensor is
// zero except at the sent indices) and of AQ-SGD (Sec. 2.5: the receiver adds
// the sent change into its copy of the per-example buffer and hands on the
// updated row).
//
// Each workgroup owns a chunk [c0, c1) of one segment's dense output.  It
// finds the payload entries that fall into its chunk (block table, else a
// cooperative search of the ascending index list), builds the chunk in LDS,
// and writes it out with full-width stores, so the dense output is written
// exactly once.  Rows of up to 2048 elements take one wavefront each
// instead.  Also here: the EF-mixed receiver (two lists, the second added),
// the EF-mixed sender's residual, and TopK at given indices (index reuse for
// gradients).
#include <algorithm>
#include <type_traits>

#include "tc_internal.hpp"
#include "tc_select.hpp"

namespace tc {

constexpr int SC_NT = 256;
constexpr int SC_VPT = 16;
constexpr uint64_t SC_CH = (uint64_t)SC_NT * SC_VPT;

// First j in [0, n) with a[j] >= c (n when none), for an ascending a.  Each
// round probes NT evenly spaced entries in parallel and keeps the gap that
// must hold the answer, so n entries take about log_{NT+1}(n) rounds.
template <int NT>
__device__ uint32_t block_lower_bound(const uint32_t* __restrict__ a, uint32_t n, uint32_t c, uint32_t* scratch) {
  uint32_t lo = 0, hi = n;
  while (lo < hi) {
    const uint64_t len = hi - lo;
    const uint32_t pt = lo + (uint32_t)(((uint64_t)(threadIdx.x + 1) * len) / (NT + 1));
    const uint32_t below = (a[pt] < c) ? 1u : 0u;
    const uint32_t cnt = block_sum<NT>(below, scratch);
    const uint32_t nlo = cnt ? lo + (uint32_t)(((uint64_t)cnt * len) / (NT + 1)) + 1u : lo;
    const uint32_t nhi = (cnt < (uint32_t)NT) ? lo + (uint32_t)(((uint64_t)(cnt + 1) * len) / (NT + 1)) : hi;
    lo = nlo;
    hi = max(nhi, nlo);   // equal bounds end the search even on unsorted input
  }
  return lo;
}

static_assert(SC_CH == BLOCK_LEN, "a receiver chunk is one block of the payload's block table");

// the payload range [j0, j1) of the chunk [c0, c1): from the block table
// when the payload carries one (checked against what a valid payload allows),
// else by searching the index list
__device__ __forceinline__ void chunk_range(const uint32_t* ix, const uint32_t* bt, uint64_t k, uint64_t c0,
                                            uint64_t c1, uint32_t* scratch, uint32_t& j0, uint32_t& j1) {
  if (bt) {
    const uint64_t c = c0 / SC_CH;
    j0 = load_uniform(bt + c);        // (c0 is the same for the whole workgroup)
    j1 = load_uniform(bt + c + 1);
    if (j0 > j1 || j1 > k || j1 - j0 > c1 - c0) {
      if (threadIdx.x == 0) raise_error(KERR_BAD_INDEX);
      j0 = j1 = 0;
    }
    return;
  }
  j0 = block_lower_bound<SC_NT>(ix, (uint32_t)k, (uint32_t)c0, scratch);
  const uint32_t rest = (uint32_t)min(k - j0, c1 - c0);
  j1 = j0 + block_lower_bound<SC_NT>(ix + j0, rest, (uint32_t)c1, scratch);
}

// MODE_VAL: wire values; MODE_CODES: b-bit codes of the kept list (one min-max
// group per segment)
enum { MODE_VAL = 0, MODE_CODES = 1 };

// Entries a chunk can hold (sorted, distinct indices inside SC_CH elements)
// spread over the threads: at most SC_VPT per thread.  Each thread loads all
// of its entries before applying any, so the loads overlap instead of paying
// one memory round trip per entry.
constexpr int SC_EPT = (int)(SC_CH / SC_NT);

template <typename WireT, typename OutT, int MODE, int B>
__global__ __launch_bounds__(SC_NT) void k_topk_scatter(ScatterArgs a) {
  using RW = typename Elem<WireT>::raw;
  using RO = typename Elem<OutT>::raw;
  __shared__ __attribute__((aligned(16))) RO buf[SC_CH];
  __shared__ uint32_t scratch[SC_NT / WAVE + 2];
  const uint64_t nch = (a.L + SC_CH - 1) / SC_CH;
  for (uint64_t wi = blockIdx.x; wi < a.n_seg * nch; wi += gridDim.x) {
    const uint64_t seg = wi / nch, c0 = (wi % nch) * SC_CH;
    const uint64_t c1 = min(a.L, c0 + SC_CH);
    const uint32_t* ix = a.idx + seg * a.k;
    const uint32_t* bt = a.blk ? a.blk + seg * (n_blocks(a.L) + 1) : nullptr;
    uint32_t j0, j1;
    chunk_range(ix, bt, a.k, c0, c1, scratch, j0, j1);
    // entries past the segment's end belong to no chunk: the last chunk flags them
    if (c1 == a.L && j1 < a.k && threadIdx.x == 0) raise_error(KERR_BAD_INDEX);
    float lo = 0.0f, scale = 0.0f;
    if constexpr (MODE == MODE_CODES) { lo = load_uniform(a.meta + 2 * seg); scale = load_uniform(a.meta + 2 * seg + 1); }
    // this thread's entries j0 + t + r*SC_NT, all loaded first
    uint32_t ei[SC_EPT];
    float ex[SC_EPT];
#pragma unroll
    for (int r = 0; r < SC_EPT; ++r) {
      const uint32_t j = j0 + threadIdx.x + (uint32_t)r * SC_NT;
      ei[r] = 0xFFFFFFFFu;
      ex[r] = 0.0f;
      if (j < j1) {
        ei[r] = ix[j];
        // without a block table the ranges come from a search that needs
        // ascending indices: check them
        if (!bt && j > j0 && ix[j - 1] >= ei[r]) raise_error(KERR_BAD_INDEX);
        if constexpr (MODE == MODE_VAL) {
          ex[r] = Elem<WireT>::up(((const RW*)a.val)[seg * a.k + j]);
        } else if constexpr (B == 32) {
          ex[r] = __uint_as_float(a.codes[seg * a.wpg + j]);
        } else {
          const uint64_t bit = (uint64_t)j * B;
          const uint32_t* w = a.codes + seg * a.wpg + (bit >> 5);
          uint32_t c = w[0] >> (bit & 31);
          if ((bit & 31) + B > 32) c |= w[1] << (32 - (bit & 31));
          c &= (1u << B) - 1u;
          const float prod = (float)c * scale;
          ex[r] = lo + prod;
        }
      }
    }
    // the chunk's part of the buffer zeroed in 16-byte pieces (a short
    // segment's chunk is the segment)
    const uint32_t nz = (uint32_t)(((c1 - c0) * sizeof(RO) + 15) / 16);
    for (uint32_t i = threadIdx.x; i < nz; i += SC_NT) reinterpret_cast<u32x4*>(buf)[i] = u32x4{0u, 0u, 0u, 0u};
    __syncthreads();
#pragma unroll
    for (int r = 0; r < SC_EPT; ++r) {
      const uint32_t j = j0 + threadIdx.x + (uint32_t)r * SC_NT;
      if (j < j1) {
        const uint32_t i = ei[r];
        if (i < c0 || i >= c1) raise_error(KERR_BAD_INDEX);
        else buf[i - c0] = Elem<OutT>::down(ex[r]);
      }
    }
    __syncthreads();
    // the dense chunk, each store instruction covering whole lines
    copy_lds_to_global<SC_NT, RO>((RO*)a.y + seg * a.L + c0, buf, (uint32_t)(c1 - c0));
    __syncthreads();
  }
}

// Receiver of short segments (token rows, at most SR_MAX elements): one
// wavefront per row and nothing shared across wavefronts, so a row costs no
// workgroup barrier and no range lookup.  The row is built in a slice of LDS
// private to the wavefront: zeroed, the row's entries written (their loads
// issued first), then stored in lane-consecutive 16-byte pieces.  Indices
// must be below L and strictly ascending; the block table is only checked.
constexpr uint32_t SR_MAX = 2048;
constexpr int SR_WAVES = SC_NT / WAVE;
static_assert(SR_MAX <= BLOCK_LEN, "a row is one block of the block table");

// A row's entries j0 + r*WAVE + lane (r < EPL), all loads issued before any
// is used: the index, the index before it (checked by the caller: indices
// ascend) and the value's bits, one register each (two 16-bit values packed
// in one register, or a use between two entries' loads, would make each
// load wait for the one before).
template <typename W>
using wire_bits_t = typename std::conditional<sizeof(W) == 4, uint32_t, uint16_t>::type;

template <int EPL, typename UW>
__device__ __forceinline__ void row_entries(const uint32_t* ix, const UW* vv, uint32_t j0, uint32_t k, uint32_t lane,
                                            uint32_t (&ei)[EPL], uint32_t (&ep)[EPL], uint32_t (&ev)[EPL]) {
  // (k >= 1: an entry at or past k reads entry 0 instead, and the caller
  // skips it; no branch stands between the loads)
#pragma unroll
  for (int r = 0; r < EPL; ++r) {
    const uint32_t j = j0 + (uint32_t)r * WAVE + lane;
    const uint32_t jj = (j < k) ? j : 0u;
    ei[r] = ix[jj];
    ev[r] = vv[jj];
    ep[r] = ix[(jj > 0u) ? jj - 1u : 0u];
  }
}

// the two block-table words of a row (a table of one block per row), or
// zeros without a table; one address either way, so that the read carries
// no branch
static __device__ const uint32_t g_no_table[2] = {0u, 0u};
__device__ __forceinline__ const uint32_t* row_table(const uint32_t* blk, uint64_t s, uint64_t L) {
  return blk ? blk + s * (n_blocks(L) + 1) : g_no_table;
}

template <typename RW>
__device__ __forceinline__ RW wire_value(uint32_t bits) {
  const wire_bits_t<RW> u = (wire_bits_t<RW>)bits;
  RW x;
  __builtin_memcpy(&x, &u, sizeof(RW));
  return x;
}

template <typename WireT, typename OutT>
__global__ __launch_bounds__(SC_NT) void k_topk_scatter_row(ScatterArgs a) {
  using RW = typename Elem<WireT>::raw;
  using RO = typename Elem<OutT>::raw;
  using UW = wire_bits_t<RW>;
  constexpr uint32_t PER = 16 / sizeof(RO);
  constexpr int EPL = 4;   // entries per lane per round, loads in flight together
  __shared__ __attribute__((aligned(16))) RO buf[SR_WAVES][SR_MAX];
  // (the wavefront's number as a scalar: a row's table words are read
  // through the scalar unit)
  const uint32_t w = (uint32_t)__builtin_amdgcn_readfirstlane((int)(threadIdx.x / WAVE)), lane = (uint32_t)lane_id();
  RO* b = buf[w];
  const uint32_t L = (uint32_t)a.L, k = (uint32_t)a.k;   // k <= L <= SR_MAX (the launcher checks)
  const bool vec = (((uintptr_t)a.y | (L * sizeof(RO))) & 15u) == 0;
  const uint64_t stride = (uint64_t)gridDim.x * SR_WAVES;
  for (uint64_t s = (uint64_t)blockIdx.x * SR_WAVES + w; s < a.n_seg; s += stride) {
    const uint32_t* ix = a.idx + s * a.k;
    const UW* vv = (const UW*)a.val + s * a.k;
    // a block table, when given, must describe the row's one block; it is
    // read with the first round of entries and checked after it
    const uint32_t* bt = row_table(a.blk, s, a.L);
    const uint32_t bt0 = load_uniform(bt), bt1 = load_uniform(bt + 1);
    uint32_t bad = 0u;
    for (uint32_t q = lane; q * PER < L; q += WAVE) reinterpret_cast<u32x4*>(b)[q] = u32x4{0u, 0u, 0u, 0u};
    for (uint32_t j0 = 0; j0 < k; j0 += EPL * WAVE) {
      uint32_t ei[EPL], ep[EPL], ev[EPL];
      row_entries<EPL>(ix, vv, j0, k, lane, ei, ep, ev);
#pragma unroll
      for (int r = 0; r < EPL; ++r) {
        const uint32_t j = j0 + (uint32_t)r * WAVE + lane;
        if (j < k) {
          if (ei[r] >= L || (j > 0 && ei[r] <= ep[r])) bad = 1u;
          else b[ei[r]] = Elem<OutT>::down(Elem<WireT>::up(wire_value<RW>(ev[r])));
        }
      }
    }
    if (a.blk && (bt0 != 0u || bt1 != k)) bad = 1u;
    if (bad) raise_error(KERR_BAD_INDEX);
    // (a wavefront's LDS accesses complete in program order)
    __builtin_amdgcn_wave_barrier();
    RO* yr = (RO*)a.y + s * a.L;
    for (uint32_t q = lane; q * PER < L; q += WAVE) {
      if (vec && q * PER + PER <= L) {
        vstore<true>(reinterpret_cast<u32x4*>(yr) + q, reinterpret_cast<const u32x4*>(b)[q]);
      } else {
        for (uint32_t c = q * PER; c < min(L, q * PER + PER); ++c) yr[c] = b[c];
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// Payload groups of eight entries, loaded with 16-byte accesses aligned in
// the whole payload array (rows of k entries need not be aligned): group g of
// a chunk covers array entries A0 + 8g .. A0 + 8g + 7.  A group reaching past
// the end of the arrays is read element by element.
template <typename R>
struct PayGroup {
  uint32_t idx[8];
  R val[8];
};

template <typename R>
__device__ __forceinline__ void load_group(const ScatterArgs& a, uint64_t Jg, uint64_t total, PayGroup<R>& g) {
  static_assert(sizeof(R) == 2, "eight 16-bit values per 16-byte access");
  if (Jg + 8 <= total) {
    const u32x4 i0 = *reinterpret_cast<const u32x4*>(a.idx + Jg);
    const u32x4 i1 = *reinterpret_cast<const u32x4*>(a.idx + Jg + 4);
    const u32x4 vv = *reinterpret_cast<const u32x4*>((const R*)a.val + Jg);
    __builtin_memcpy(g.idx, &i0, 16);
    __builtin_memcpy(g.idx + 4, &i1, 16);
    __builtin_memcpy(g.val, &vv, 16);
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint64_t J = Jg + e;
      g.idx[e] = (J < total) ? a.idx[J] : 0u;
      g.val[e] = (J < total) ? ((const R*)a.val)[J] : R{};
    }
  }
}

// apply the group's entries that lie in [J0, J1) to the chunk [c0, c1) held
// in LDS: buf[i - c0] = out(in(buf[i - c0]) + in(val)); an index outside the
// chunk is flagged
template <typename T>
__device__ __forceinline__ void apply_group(const PayGroup<typename Elem<T>::raw>& g, uint64_t Jg, uint64_t J0,
                                            uint64_t J1, uint64_t c0, uint64_t c1, typename Elem<T>::raw* buf) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint64_t J = Jg + e;
    if (J >= J0 && J < J1) {
      const uint32_t i = g.idx[e];
      if (i < c0 || i >= c1) raise_error(KERR_BAD_INDEX);
      else buf[i - c0] = Elem<T>::down(Elem<T>::up(buf[i - c0]) + Elem<T>::up(g.val[e]));
    }
  }
}

// AQ-SGD receiver.  Workgroup = one 4096-element chunk of one example's row.
// The example id and the chunk's payload range are read first, together;
// then the row chunk (m_r) and the chunk's payload entries are loaded at the
// same time; the row goes to LDS, the entries are applied there, and the
// updated chunk is written to m_r and to a_hat with full-line stores.
template <typename T>
__global__ __launch_bounds__(SC_NT) void k_aqsgd_recv(ScatterArgs a) {
  using R = typename Elem<T>::raw;
  constexpr int PER = 16 / (int)sizeof(R);            // elements per 16-byte access
  constexpr int VPT = (int)(SC_CH / SC_NT);           // elements per thread
  constexpr int GPT = 2;                              // payload groups per thread held in registers
  static_assert(VPT % PER == 0, "whole 16-byte runs per thread");
  __shared__ __attribute__((aligned(16))) R buf[SC_CH];
  __shared__ uint32_t scratch[SC_NT / WAVE + 2];
  const uint64_t nch = (a.L + SC_CH - 1) / SC_CH;
  const uint64_t nbt = n_blocks(a.L) + 1;
  // 16-byte paths: 16-bit data, 16-byte aligned rows and payload arrays, a block table
  const bool vec = sizeof(R) == 2 && (a.L % 8) == 0 && a.blk != nullptr &&
                   (((uintptr_t)a.m | (uintptr_t)a.y | (uintptr_t)a.idx | (uintptr_t)a.val) & 15u) == 0;
  const uint64_t total = a.n_seg * a.k;
  for (uint64_t wi = blockIdx.x; wi < a.n_seg * nch; wi += gridDim.x) {
    const uint64_t b = wi / nch, ci = wi % nch, c0 = ci * SC_CH;
    const uint64_t c1 = min(a.L, c0 + SC_CH);
    // the id and (with a block table) the payload range, in one round trip
    // of the scalar unit
    const int64_t id = load_uniform(a.ids + b);
    uint32_t bj0 = 0, bj1 = 0;
    if (a.blk) { bj0 = load_uniform(a.blk + b * nbt + ci); bj1 = load_uniform(a.blk + b * nbt + ci + 1); }
    if (id < 0 || (uint64_t)id >= a.n_samples) {
      if (threadIdx.x == 0) raise_error(KERR_BAD_ID);
      continue;
    }
    R* row = (R*)a.m + (uint64_t)id * a.L;
    R* out = (R*)a.y + b * a.L;
    const bool full = vec && c1 - c0 == SC_CH;
    const uint64_t t0 = c0 + (uint64_t)threadIdx.x * VPT;
    const int nv = (int)min((uint64_t)VPT, sat_sub(c1, t0));
    R mr[VPT];
    uint32_t j0 = 0, j1 = 0;
    bool range_ok = true;
    bool done = false;
    if constexpr (sizeof(R) == 2) {
     if (full) {
      done = true;
      // row chunk and payload groups, all loads in flight together; the
      // row in lane-consecutive 16-byte pieces (piece q * SC_NT + thread:
      // whole lines per wavefront access)
#pragma unroll
      for (int q = 0; q < VPT / PER; ++q) {
        const u32x4 w = vload<true>(reinterpret_cast<const u32x4*>(row + c0) + q * SC_NT + threadIdx.x);
        __builtin_memcpy(&mr[q * PER], &w, 16);
      }
      j0 = bj0;
      j1 = bj1;
      range_ok = !(j0 > j1 || j1 > a.k || j1 - j0 > c1 - c0);
      if (!range_ok) j0 = j1 = 0;
      const uint64_t J0 = b * a.k + j0, J1 = b * a.k + j1, A0 = J0 & ~7ull;
      const uint32_t ng = (uint32_t)((J1 - A0 + 7) / 8);
      PayGroup<R> pg[GPT];
#pragma unroll
      for (int r = 0; r < GPT; ++r) {
        const uint32_t gq = threadIdx.x + (uint32_t)r * SC_NT;
        if (gq < ng) load_group<R>(a, A0 + 8ull * gq, total, pg[r]);
      }
#pragma unroll
      for (int q = 0; q < VPT / PER; ++q) {
        u32x4 w;
        __builtin_memcpy(&w, &mr[q * PER], 16);
        reinterpret_cast<u32x4*>(buf)[q * SC_NT + threadIdx.x] = w;
      }
      __syncthreads();
      // the held groups' entries: every read of the chunk goes out before
      // any write (a chunk's indices are distinct), one LDS round trip
      // rather than one per entry
      R old[GPT][8];
#pragma unroll
      for (int r = 0; r < GPT; ++r) {
        const uint32_t gq = threadIdx.x + (uint32_t)r * SC_NT;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint64_t J = A0 + 8ull * gq + (uint64_t)e;
          const uint32_t i = pg[r].idx[e];
          old[r][e] = R{};
          if (gq < ng && J >= J0 && J < J1 && i >= c0 && i < c1) old[r][e] = buf[i - c0];
        }
      }
#pragma unroll
      for (int r = 0; r < GPT; ++r) {
        const uint32_t gq = threadIdx.x + (uint32_t)r * SC_NT;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint64_t J = A0 + 8ull * gq + (uint64_t)e;
          if (gq < ng && J >= J0 && J < J1) {
            const uint32_t i = pg[r].idx[e];
            if (i < c0 || i >= c1) raise_error(KERR_BAD_INDEX);
            else buf[i - c0] = Elem<T>::down(Elem<T>::up(old[r][e]) + Elem<T>::up(pg[r].val[e]));
          }
        }
      }
      // a chunk with more entries than the registers hold: the rest in turns
      for (uint32_t gq = threadIdx.x + GPT * SC_NT; gq < ng; gq += SC_NT) {
        PayGroup<R> g1;
        load_group<R>(a, A0 + 8ull * gq, total, g1);
        apply_group<T>(g1, A0 + 8ull * gq, J0, J1, c0, c1, buf);
      }
     }
    }
    if (!done) {
      if (nv > 0) load_run_partial<R, VPT, false>(row + t0, nv, R{}, mr);
      const uint32_t* ix = a.idx + b * a.k;
      const uint32_t* bt = a.blk ? a.blk + b * nbt : nullptr;
      chunk_range(ix, bt, a.k, c0, c1, scratch, j0, j1);
      if (nv > 0) store_run<R, VPT>(&buf[threadIdx.x * VPT], mr);
      __syncthreads();
      for (uint32_t j = j0 + threadIdx.x; j < j1; j += SC_NT) {
        const uint32_t i = ix[j];
        if (!bt && j > j0 && ix[j - 1] >= i) raise_error(KERR_BAD_INDEX);
        if (i < c0 || i >= c1) raise_error(KERR_BAD_INDEX);
        else buf[i - c0] = Elem<T>::down(Elem<T>::up(buf[i - c0]) + Elem<T>::up(((const R*)a.val)[b * a.k + j]));
      }
    }
    if (!range_ok && threadIdx.x == 0) raise_error(KERR_BAD_INDEX);
    if (c1 == a.L && j1 < a.k && threadIdx.x == 0) raise_error(KERR_BAD_INDEX);
    __syncthreads();
    // the updated row chunk to the buffer and to a_hat in lane-consecutive
    // 16-byte pieces (whole lines per wavefront store)
    if (full) {
#pragma unroll
      for (int q = 0; q < VPT / PER; ++q) {
        const uint32_t pc = (uint32_t)q * SC_NT + threadIdx.x;
        const u32x4 w = reinterpret_cast<const u32x4*>(buf)[pc];
        vstore<true>(reinterpret_cast<u32x4*>(row + c0) + pc, w);
        vstore<true>(reinterpret_cast<u32x4*>(out + c0) + pc, w);
      }
    } else {
      copy_lds_to_global<SC_NT, R>(row + c0, buf, (uint32_t)(c1 - c0));
      copy_lds_to_global<SC_NT, R>(out + c0, buf, (uint32_t)(c1 - c0));
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------- EF-mixed
// Receiver of EF-mixed (Sec. 2.4): the dense tensor starts at +0, takes the
// input list's values at its indices, then adds the error buffer's list at
// its indices (binary32; the two lists may share indices), and is rounded
// once to the output dtype.  Workgroup iteration = one 4096-element chunk of
// one segment, built in LDS as binary32; each list's range in the chunk comes
// from its block table, else from a search of its ascending indices.
template <typename WireT, typename OutT>
__global__ __launch_bounds__(SC_NT) void k_efmix_scatter(ScatterArgs a) {
  using RW = typename Elem<WireT>::raw;
  using RO = typename Elem<OutT>::raw;
  __shared__ __attribute__((aligned(16))) float buf[SC_CH];
  __shared__ uint32_t scratch[SC_NT / WAVE + 2];
  const uint64_t nch = (a.L + SC_CH - 1) / SC_CH;
  const uint64_t nbt = n_blocks(a.L) + 1;
  const uint32_t t = threadIdx.x;
  for (uint64_t wi = blockIdx.x; wi < a.n_seg * nch; wi += gridDim.x) {
    const uint64_t seg = wi / nch, c0 = (wi % nch) * SC_CH;
    const uint64_t c1 = min(a.L, c0 + SC_CH);
    const uint32_t n = (uint32_t)(c1 - c0);
    const uint64_t kk[2] = {a.k, a.k2};
    const uint32_t* ixl[2] = {a.idx + seg * a.k, a.idx2 + seg * a.k2};
    const uint32_t* btl[2] = {a.blk ? a.blk + seg * nbt : nullptr, a.blk2 ? a.blk2 + seg * nbt : nullptr};
    const RW* vl[2] = {(const RW*)a.val + seg * a.k, (const RW*)a.val2 + seg * a.k2};
    // both lists' ranges in the chunk (block tables: one round trip for both)
    uint32_t r0[2] = {0u, 0u}, r1[2] = {0u, 0u};
    if (btl[0] && btl[1]) {
      const uint64_t c = c0 / SC_CH;
#pragma unroll
      for (int l = 0; l < 2; ++l) { r0[l] = load_uniform(btl[l] + c); r1[l] = load_uniform(btl[l] + c + 1); }
#pragma unroll
      for (int l = 0; l < 2; ++l) {
        if (r0[l] > r1[l] || r1[l] > kk[l] || r1[l] - r0[l] > n) {
          if (t == 0) raise_error(KERR_BAD_INDEX);
          r0[l] = r1[l] = 0u;
        }
      }
    } else {
#pragma unroll
      for (int l = 0; l < 2; ++l)
        if (kk[l] > 0) chunk_range(ixl[l], btl[l], kk[l], c0, c1, scratch, r0[l], r1[l]);
    }
    // entries past the segment's end belong to no chunk: the last chunk flags them
#pragma unroll
    for (int l = 0; l < 2; ++l)
      if (c1 == a.L && r1[l] < kk[l] && t == 0) raise_error(KERR_BAD_INDEX);
    // this thread's first entry of each list, both loaded together
    uint32_t fi[2];
    float fv[2];
#pragma unroll
    for (int l = 0; l < 2; ++l) {
      const uint32_t j = r0[l] + t;
      fi[l] = (j < r1[l]) ? ixl[l][j] : 0u;
      fv[l] = (j < r1[l]) ? Elem<WireT>::up(vl[l][j]) : 0.0f;
    }
    for (uint32_t q = t; q * 4 < n; q += SC_NT) reinterpret_cast<u32x4*>(buf)[q] = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int l = 0; l < 2; ++l) {
      __syncthreads();   // the zeroed chunk, then the first list, are in place
      for (uint32_t j = r0[l] + t; j < r1[l]; j += SC_NT) {
        const bool first = j == r0[l] + t;
        const uint32_t i = first ? fi[l] : ixl[l][j];
        const float v = first ? fv[l] : Elem<WireT>::up(vl[l][j]);
        if (!btl[l] && j > r0[l] && ixl[l][j - 1] >= i) raise_error(KERR_BAD_INDEX);
        if (i < c0 || i >= c1) raise_error(KERR_BAD_INDEX);
        else buf[i - c0] = l ? buf[i - c0] + v : v;
      }
    }
    __syncthreads();
    // rounded to the output dtype, in lane-consecutive pieces of four
    RO* yc = (RO*)a.y + seg * a.L + c0;
    for (uint32_t q = t; q * 4 < n; q += SC_NT) {
      const int nv = (int)min(4u, n - q * 4);
      RO o[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) o[c] = Elem<OutT>::down(buf[q * 4 + c]);
      store_run_partial<RO, 4, true>(yc + q * 4, nv, o);
    }
    __syncthreads();
  }
}

// EF-mixed residual (Sec. 2.4), the sender's second kernel, after both
// selections: e <- (x minus what was sent of it) + (e minus what was sent
// of it).  x is exact in its dtype, so its share is x off the input's list
// and +0 on it.  Where both lists hold an index the receiver rounds
// u = x + wire(e) (binary32) once to the wire dtype, and the part that
// rounding drops, u - wire(u), stays in the buffer too.  Workgroup
// iteration = one 4096-element chunk: its x and e are loaded first
// (lane-consecutive pieces of four), both lists' entries in the chunk set
// bits of two LDS masks (ranges from the block tables, else a search of the
// ascending indices), then e is written in the same pieces.
template <typename InT>
__global__ __launch_bounds__(SC_NT) void k_efmix_resid(EfmixResidArgs a) {
  using R = typename Elem<InT>::raw;
  constexpr int QPT = (int)(SC_CH / 4 / SC_NT);   // pieces per thread
  __shared__ uint32_t msk[2][SC_CH / 32];
  __shared__ uint32_t scratch[SC_NT / WAVE + 2];
  const uint64_t nch = (a.L + SC_CH - 1) / SC_CH;
  const uint64_t nbt = n_blocks(a.L) + 1;
  const uint32_t t = threadIdx.x;
  const bool vec = ((((uintptr_t)a.x | (uintptr_t)a.e) & 15u) == 0) && (a.L % 4u) == 0;
  for (uint64_t wi = blockIdx.x; wi < a.n_seg * nch; wi += gridDim.x) {
    const uint64_t seg = wi / nch, c0 = (wi % nch) * SC_CH;
    const uint64_t c1 = min(a.L, c0 + SC_CH);
    const uint32_t n = (uint32_t)(c1 - c0);
    const R* xc = (const R*)a.x + seg * a.L + c0;
    float* ec = a.e + seg * a.L + c0;
    R xr[QPT][4];
    float er[QPT][4];
    auto load_chunk = [&](auto vec_c) {
      constexpr bool VEC = decltype(vec_c)::value;
#pragma unroll
      for (int q = 0; q < QPT; ++q) {
        const uint32_t i0 = ((uint32_t)q * SC_NT + t) * 4;
        if constexpr (VEC) {
          // (vec: pieces aligned and whole; one past the chunk's end reads
          // the chunk's first piece, unused, so that no branch stands
          // between the loads)
          const uint32_t ia = (i0 < n) ? i0 : 0u;
          load_piece<R, true>(xc + ia, xr[q]);
          load_piece<float, true>(ec + ia, er[q]);
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            xr[q][c] = (i0 + (uint32_t)c < n) ? xc[i0 + c] : R{};
            er[q][c] = (i0 + (uint32_t)c < n) ? ec[i0 + c] : 0.0f;
          }
        }
      }
    };
    if (vec) load_chunk(std::true_type{});
    else load_chunk(std::false_type{});
    const uint64_t kk[2] = {a.k, a.k2};
    const uint32_t* ixl[2] = {a.idx + seg * a.k, a.idx2 + seg * a.k2};
    const uint32_t* btl[2] = {a.blk ? a.blk + seg * nbt : nullptr, a.blk2 ? a.blk2 + seg * nbt : nullptr};
    for (uint32_t i = t; i < 2 * (SC_CH / 32); i += SC_NT) (&msk[0][0])[i] = 0u;
    // both lists' ranges in the chunk (block tables: one round trip for both)
    uint32_t r0[2] = {0u, 0u}, r1[2] = {0u, 0u};
    if (btl[0] && btl[1]) {
      const uint64_t c = c0 / SC_CH;
#pragma unroll
      for (int l = 0; l < 2; ++l) { r0[l] = load_uniform(btl[l] + c); r1[l] = load_uniform(btl[l] + c + 1); }
#pragma unroll
      for (int l = 0; l < 2; ++l) {
        if (r0[l] > r1[l] || r1[l] > kk[l] || r1[l] - r0[l] > n) {
          if (t == 0) raise_error(KERR_BAD_INDEX);
          r0[l] = r1[l] = 0u;
        }
      }
    } else {
#pragma unroll
      for (int l = 0; l < 2; ++l)
        if (kk[l] > 0) chunk_range(ixl[l], btl[l], kk[l], c0, c1, scratch, r0[l], r1[l]);
    }
    // entries past the segment's end belong to no chunk: the last chunk flags them
#pragma unroll
    for (int l = 0; l < 2; ++l)
      if (c1 == a.L && r1[l] < kk[l] && t == 0) raise_error(KERR_BAD_INDEX);
    __syncthreads();   // the zeroed masks
#pragma unroll
    for (int l = 0; l < 2; ++l) {
      for (uint32_t j = r0[l] + t; j < r1[l]; j += SC_NT) {
        const uint32_t i = ixl[l][j];
        if (!btl[l] && j > r0[l] && ixl[l][j - 1] >= i) raise_error(KERR_BAD_INDEX);
        if (i < c0 || i >= c1) raise_error(KERR_BAD_INDEX);
        else atomicOr(&msk[l][(i - c0) >> 5], 1u << ((i - c0) & 31u));
      }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < QPT; ++q) {
      const uint32_t i0 = ((uint32_t)q * SC_NT + t) * 4;
      if (i0 >= n) continue;
      const uint32_t kx4 = msk[0][i0 >> 5] >> (i0 & 31u), ke4 = msk[1][i0 >> 5] >> (i0 & 31u);
      float o[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float xv = Elem<InT>::up(xr[q][c]);
        const bool in_x = (kx4 >> c) & 1u, in_e = (ke4 >> c) & 1u;
        const float rx = xv - (in_x ? xv : 0.0f);
        const float v = er[q][c];
        const float ve = through<InT>(v);
        float re = v - (in_e ? ve : 0.0f);
        if (in_x && in_e) {
          const float u = xv + ve;
          re = re + (u - through<InT>(u));
        }
        o[c] = rx + re;
      }
      if (vec && i0 + 4 <= n) {
        store_run<float, 4, true>(ec + i0, o);
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c)
          if (i0 + (uint32_t)c < n) ec[i0 + c] = o[c];
      }
    }
    __syncthreads();   // the masks are cleared for the next chunk
  }
}

// AQ-SGD receiver for rows of up to SR_MAX elements (one buffer row per
// token row): one wavefront per row, in a slice of LDS of its own.  The row's
// payload entries do not depend on the id, so they are loaded with the id;
// the buffer row follows, goes to LDS, takes the entries (a read-modify-write
// per entry: the indices of a valid row are distinct) and leaves for m_r and
// a_hat in lane-consecutive 16-byte pieces.
template <typename T>
__global__ __launch_bounds__(SC_NT) void k_aqsgd_recv_row(ScatterArgs a) {
  using R = typename Elem<T>::raw;
  using UW = wire_bits_t<R>;
  constexpr uint32_t PER = 16 / sizeof(R);
  constexpr int EPL = 4;   // entries per lane per round
  __shared__ __attribute__((aligned(16))) R buf[SR_WAVES][SR_MAX];
  // (the wavefront's number as a scalar: a row's id and table words are read
  // through the scalar unit)
  const uint32_t w = (uint32_t)__builtin_amdgcn_readfirstlane((int)(threadIdx.x / WAVE)), lane = (uint32_t)lane_id();
  R* b = buf[w];
  const uint32_t L = (uint32_t)a.L, k = (uint32_t)a.k;   // k <= L <= SR_MAX (the launcher checks)
  const bool vec = (((uintptr_t)a.m | (uintptr_t)a.y | (L * sizeof(R))) & 15u) == 0;
  const uint64_t stride = (uint64_t)gridDim.x * SR_WAVES;
  for (uint64_t s = (uint64_t)blockIdx.x * SR_WAVES + w; s < a.n_seg; s += stride) {
    const uint32_t* ix = a.idx + s * a.k;
    const UW* vv = (const UW*)a.val + s * a.k;
    const int64_t id = load_uniform(a.ids + s);
    // the first round of entries, and the block table's two words, go out
    // with the id
    const uint32_t* bt = row_table(a.blk, s, a.L);
    const uint32_t bt0 = load_uniform(bt), bt1 = load_uniform(bt + 1);
    uint32_t ei[EPL], ep[EPL], ev[EPL];
    if (k > 0) row_entries<EPL>(ix, vv, 0u, k, lane, ei, ep, ev);
    if (id < 0 || (uint64_t)id >= a.n_samples) {
      if (lane == 0) raise_error(KERR_BAD_ID);
      continue;
    }
    uint32_t bad = (a.blk && (bt0 != 0u || bt1 != k)) ? 1u : 0u;
    R* row = (R*)a.m + (uint64_t)id * a.L;
    for (uint32_t q = lane; q * PER < L; q += WAVE) {
      if (vec && q * PER + PER <= L) {
        reinterpret_cast<u32x4*>(b)[q] = vload<true>(reinterpret_cast<const u32x4*>(row) + q);
      } else {
        for (uint32_t c = q * PER; c < min(L, q * PER + PER); ++c) b[c] = row[c];
      }
    }
    // (a wavefront's LDS accesses complete in program order)
    for (uint32_t j0 = 0; j0 < k; j0 += EPL * WAVE) {
      if (j0 > 0) row_entries<EPL>(ix, vv, j0, k, lane, ei, ep, ev);
#pragma unroll
      for (int r = 0; r < EPL; ++r) {
        const uint32_t j = j0 + (uint32_t)r * WAVE + lane;
        if (j < k) {
          if (ei[r] >= L || (j > 0 && ei[r] <= ep[r])) bad = 1u;
          else b[ei[r]] = Elem<T>::down(Elem<T>::up(b[ei[r]]) + Elem<T>::up(wire_value<R>(ev[r])));
        }
      }
    }
    if (bad) raise_error(KERR_BAD_INDEX);
    __builtin_amdgcn_wave_barrier();
    R* out = (R*)a.y + s * a.L;
    for (uint32_t q = lane; q * PER < L; q += WAVE) {
      if (vec && q * PER + PER <= L) {
        const u32x4 v4 = reinterpret_cast<const u32x4*>(b)[q];
        vstore<true>(reinterpret_cast<u32x4*>(row) + q, v4);
        vstore<true>(reinterpret_cast<u32x4*>(out) + q, v4);
      } else {
        for (uint32_t c = q * PER; c < min(L, q * PER + PER); ++c) {
          row[c] = b[c];
          out[c] = b[c];
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// ---------------------------------------------------------- index reuse
// TopK at given indices (Sec. 3.2: in the GPT-2 runs the gradients are
// compressed at the indices that the activations' TopK kept).  The message
// is x at those indices in x's own dtype; without error feedback every entry
// is independent.  An index outside the segment sends +0 and is flagged.
template <typename T>
__global__ __launch_bounds__(SC_NT) void k_gather(GatherArgs a) {
  using R = typename Elem<T>::raw;
  const uint64_t total = a.n_seg * a.k;
  for (uint64_t g = (uint64_t)blockIdx.x * SC_NT + threadIdx.x; g < total; g += (uint64_t)gridDim.x * SC_NT) {
    const uint64_t s = g / a.k;
    const uint32_t i = a.idx[g];
    R v = R{};
    if (i < a.L) v = ((const R*)a.x)[s * a.L + i];
    else raise_error(KERR_BAD_INDEX);
    ((R*)a.val)[g] = v;
  }
}

// With error feedback (Sec. 2.4): X = x + e is compressed and e becomes X
// minus what the receiver holds, so the whole residual is rewritten.  One
// 4096-element chunk per iteration: X into LDS, the chunk's entries (range
// from the block table, else a search of the ascending indices) send X and
// mark their places, then the residual leaves densely.
template <typename T>
__global__ __launch_bounds__(SC_NT) void k_gather_ef(GatherArgs a) {
  using R = typename Elem<T>::raw;
  __shared__ float s_x[SC_CH];
  __shared__ uint8_t s_f[SC_CH];
  __shared__ uint32_t scratch[SC_NT / WAVE + 2];
  const uint64_t nch = (a.L + SC_CH - 1) / SC_CH;
  const uint64_t nbt = n_blocks(a.L) + 1;
  const uint32_t t = threadIdx.x;
  for (uint64_t wi = blockIdx.x; wi < a.n_seg * nch; wi += gridDim.x) {
    const uint64_t seg = wi / nch, c0 = (wi % nch) * SC_CH;
    const uint64_t c1 = min(a.L, c0 + SC_CH);
    const uint32_t* ix = a.idx + seg * a.k;
    const uint32_t* bt = a.blk ? a.blk + seg * nbt : nullptr;
    uint32_t j0 = 0, j1 = 0;
    if (a.k > 0) chunk_range(ix, bt, a.k, c0, c1, scratch, j0, j1);
    // entries past the segment's end belong to no chunk: the last chunk flags them
    if (c1 == a.L && j1 < a.k && t == 0) raise_error(KERR_BAD_INDEX);
    // X = x + e, thread-contiguous runs
    const uint64_t t0 = c0 + (uint64_t)t * SC_VPT;
    const int nv = (int)min((uint64_t)SC_VPT, sat_sub(c1, t0));
    R xr[SC_VPT];
    float er[SC_VPT];
    if (nv > 0) {
      load_run_partial<R, SC_VPT, false>((const R*)a.x + seg * a.L + t0, nv, R{}, xr);
      load_run_partial<float, SC_VPT, false>(a.e + seg * a.L + t0, nv, 0.0f, er);
    }
#pragma unroll
    for (int i = 0; i < SC_VPT; ++i) {
      s_x[t * SC_VPT + i] = (i < nv) ? Elem<T>::up(xr[i]) + er[i] : 0.0f;
      s_f[t * SC_VPT + i] = 0;
    }
    __syncthreads();
    for (uint32_t j = j0 + t; j < j1; j += SC_NT) {
      const uint32_t i = ix[j];
      if (!bt && j > j0 && ix[j - 1] >= i) raise_error(KERR_BAD_INDEX);
      if (i < c0 || i >= c1) {
        raise_error(KERR_BAD_INDEX);
        ((R*)a.val)[seg * a.k + j] = R{};
      } else {
        ((R*)a.val)[seg * a.k + j] = Elem<T>::down(s_x[i - c0]);
        s_f[i - c0] = 1;
      }
    }
    __syncthreads();
    if (nv > 0) {
      float o[SC_VPT];
#pragma unroll
      for (int i = 0; i < SC_VPT; ++i) {
        const float X = s_x[t * SC_VPT + i];
        o[i] = X - (s_f[t * SC_VPT + i] ? through<T>(X) : 0.0f);
      }
      store_run_partial<float, SC_VPT, false>(a.e + seg * a.L + t0, nv, o);
    }
    __syncthreads();
  }
}

namespace {

uint32_t scatter_grid(uint64_t n_seg, uint64_t L) {
  const uint64_t work = n_seg * ((L + SC_CH - 1) / SC_CH);
  return (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(work, (uint64_t)device_cus() * 8));
}

template <typename WireT>
const void* val_ptr(int out_dt) {
  if (out_dt == DT_F32) return (const void*)k_topk_scatter<WireT, float, MODE_VAL, 0>;
  if (out_dt == DT_BF16) return (const void*)k_topk_scatter<WireT, bf16_t, MODE_VAL, 0>;
  return (const void*)k_topk_scatter<WireT, f16_t, MODE_VAL, 0>;
}

template <typename WireT>
const void* row_ptr(int out_dt) {
  if (out_dt == DT_F32) return (const void*)k_topk_scatter_row<WireT, float>;
  if (out_dt == DT_BF16) return (const void*)k_topk_scatter_row<WireT, bf16_t>;
  return (const void*)k_topk_scatter_row<WireT, f16_t>;
}

template <typename OutT>
const void* codes_ptr(uint32_t b) {
  switch (b) {
    case 1: return (const void*)k_topk_scatter<float, OutT, MODE_CODES, 1>;
    case 2: return (const void*)k_topk_scatter<float, OutT, MODE_CODES, 2>;
    case 3: return (const void*)k_topk_scatter<float, OutT, MODE_CODES, 3>;
    case 4: return (const void*)k_topk_scatter<float, OutT, MODE_CODES, 4>;
    case 5: return (const void*)k_topk_scatter<float, OutT, MODE_CODES, 5>;
    case 6: return (const void*)k_topk_scatter<float, OutT, MODE_CODES, 6>;
    case 7: return (const void*)k_topk_scatter<float, OutT, MODE_CODES, 7>;
    case 8: return (const void*)k_topk_scatter<float, OutT, MODE_CODES, 8>;
    case 32: return (const void*)k_topk_scatter<float, OutT, MODE_CODES, 32>;
  }
  return nullptr;
}

}  // namespace

// wire < 0 selects the quantized kept list (bits = -wire)
hipError_t launch_topk_decompress(int wire, int out_dt, const ScatterArgs& args, hipStream_t st) {
  const void* fn = nullptr;
  if (wire >= 0) {
    fn = (wire == DT_F32) ? val_ptr<float>(out_dt) : (wire == DT_BF16) ? val_ptr<bf16_t>(out_dt) : val_ptr<f16_t>(out_dt);
  } else {
    const uint32_t b = (uint32_t)(-wire);
    fn = (out_dt == DT_F32) ? codes_ptr<float>(b) : (out_dt == DT_BF16) ? codes_ptr<bf16_t>(b) : codes_ptr<f16_t>(b);
  }
  if (!fn) return hipErrorInvalidValue;
  ScatterArgs a = args;
  void* params[] = {&a};
  if (wire >= 0 && a.L <= SR_MAX) {
    // one wavefront per row
    const void* fr = (wire == DT_F32) ? row_ptr<float>(out_dt) : (wire == DT_BF16) ? row_ptr<bf16_t>(out_dt)
                                                                                  : row_ptr<f16_t>(out_dt);
    const uint64_t wgs = (a.n_seg + SR_WAVES - 1) / SR_WAVES;
    const uint32_t grid = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(wgs, (uint64_t)device_cus() * 8));
    return hipLaunchKernel(fr, dim3(grid), dim3(SC_NT), params, 0, st);
  }
  return hipLaunchKernel(fn, dim3(scatter_grid(a.n_seg, a.L)), dim3(SC_NT), params, 0, st);
}

template <typename WireT>
const void* efmix_ptr(int out_dt) {
  if (out_dt == DT_F32) return (const void*)k_efmix_scatter<WireT, float>;
  if (out_dt == DT_BF16) return (const void*)k_efmix_scatter<WireT, bf16_t>;
  return (const void*)k_efmix_scatter<WireT, f16_t>;
}

hipError_t launch_efmix_recv(int wire, int out_dt, const ScatterArgs& args, hipStream_t st) {
  const void* fn = (wire == DT_F32) ? efmix_ptr<float>(out_dt)
                 : (wire == DT_BF16) ? efmix_ptr<bf16_t>(out_dt) : efmix_ptr<f16_t>(out_dt);
  ScatterArgs a = args;
  void* params[] = {&a};
  return hipLaunchKernel(fn, dim3(scatter_grid(a.n_seg, a.L)), dim3(SC_NT), params, 0, st);
}

hipError_t launch_efmix_resid(int dt, const EfmixResidArgs& args, hipStream_t st) {
  const void* fn = (dt == DT_F32) ? (const void*)k_efmix_resid<float>
                 : (dt == DT_BF16) ? (const void*)k_efmix_resid<bf16_t> : (const void*)k_efmix_resid<f16_t>;
  EfmixResidArgs a = args;
  void* params[] = {&a};
  return hipLaunchKernel(fn, dim3(scatter_grid(a.n_seg, a.L)), dim3(SC_NT), params, 0, st);
}

hipError_t launch_aqsgd_recv(int dt, const ScatterArgs& args, hipStream_t st) {
  ScatterArgs a = args;
  void* params[] = {&a};
  if (a.L <= SR_MAX) {
    // one wavefront per row
    const void* fr = (dt == DT_F32) ? (const void*)k_aqsgd_recv_row<float>
                   : (dt == DT_BF16) ? (const void*)k_aqsgd_recv_row<bf16_t> : (const void*)k_aqsgd_recv_row<f16_t>;
    const uint64_t wgs = (a.n_seg + SR_WAVES - 1) / SR_WAVES;
    const uint32_t grid = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(wgs, (uint64_t)device_cus() * 8));
    return hipLaunchKernel(fr, dim3(grid), dim3(SC_NT), params, 0, st);
  }
  const void* fn = (dt == DT_F32) ? (const void*)k_aqsgd_recv<float>
                 : (dt == DT_BF16) ? (const void*)k_aqsgd_recv<bf16_t> : (const void*)k_aqsgd_recv<f16_t>;
  return hipLaunchKernel(fn, dim3(scatter_grid(a.n_seg, a.L)), dim3(SC_NT), params, 0, st);
}

// The same for rows of up to SR_MAX elements (token rows): one wavefront per
// row in a slice of LDS of its own.  The row's indices are loaded first (they
// do not depend on the data), X = x + e goes to the slice in lane-consecutive
// pieces, each entry sends X and leaves X minus its wire value in the slice,
// and the slice leaves as the new residual.
template <typename T>
__global__ __launch_bounds__(SC_NT) void k_gather_ef_row(GatherArgs a) {
  using R = typename Elem<T>::raw;
  constexpr int EPL = 4;   // entries per lane per round
  __shared__ __attribute__((aligned(16))) float buf[SR_WAVES][SR_MAX];
  // (the wavefront's number as a scalar: a row's table words are read
  // through the scalar unit)
  const uint32_t w = (uint32_t)__builtin_amdgcn_readfirstlane((int)(threadIdx.x / WAVE)), lane = (uint32_t)lane_id();
  float* b = buf[w];
  const uint32_t L = (uint32_t)a.L, k = (uint32_t)a.k;   // k <= L <= SR_MAX (the launcher checks)
  const bool vec = ((((uintptr_t)a.x | (uintptr_t)a.e) & 15u) == 0) && (L % 4u) == 0;
  const uint64_t stride = (uint64_t)gridDim.x * SR_WAVES;
  for (uint64_t s = (uint64_t)blockIdx.x * SR_WAVES + w; s < a.n_seg; s += stride) {
    const uint32_t* ix = a.idx + s * a.k;
    R* vo = (R*)a.val + s * a.k;
    const R* xs = (const R*)a.x + s * a.L;
    float* es = a.e + s * a.L;
    // a block table, when given, must describe the row's one block; it is
    // read with the first loads and checked after the entries
    const uint32_t* bt = row_table(a.blk, s, a.L);
    const uint32_t bt0 = load_uniform(bt), bt1 = load_uniform(bt + 1);
    uint32_t bad = 0u;
    // X = x + e into the slice, four elements per piece, a round of four
    // pieces per lane loaded before any is used (vec: a piece past the
    // row's end reads the first piece, unused)
    constexpr int PPL = 4;
    for (uint32_t q0 = 0; q0 * 4 < L; q0 += PPL * WAVE) {
      if (vec) {
        R xr[PPL][4];
        float er[PPL][4];
#pragma unroll
        for (int p = 0; p < PPL; ++p) {
          const uint32_t q = q0 + (uint32_t)p * WAVE + lane;
          const uint32_t qa = (q * 4 < L) ? q : 0u;
          load_piece<R, true>(xs + qa * 4, xr[p]);
          load_piece<float, true>(es + qa * 4, er[p]);
        }
#pragma unroll
        for (int p = 0; p < PPL; ++p) {
          const uint32_t q = q0 + (uint32_t)p * WAVE + lane;
          if (q * 4 < L) {
            float o[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) o[c] = Elem<T>::up(xr[p][c]) + er[p][c];
            u32x4 v4;
            __builtin_memcpy(&v4, o, 16);
            reinterpret_cast<u32x4*>(b)[q] = v4;
          }
        }
      } else {
        for (uint32_t q = q0 + lane; q < q0 + PPL * WAVE && q * 4 < L; q += WAVE)
          for (uint32_t c = q * 4; c < min(L, q * 4 + 4); ++c) b[c] = Elem<T>::up(xs[c]) + es[c];
      }
    }
    // (a wavefront's LDS accesses complete in program order)
    for (uint32_t j0 = 0; j0 < k; j0 += EPL * WAVE) {
      // (k >= 1: an entry at or past k reads entry 0 and is skipped; no
      // branch stands between the loads)
      uint32_t ei[EPL], ep[EPL];
#pragma unroll
      for (int r = 0; r < EPL; ++r) {
        const uint32_t j = j0 + (uint32_t)r * WAVE + lane;
        const uint32_t jj = (j < k) ? j : 0u;
        ei[r] = ix[jj];
        ep[r] = ix[(jj > 0u) ? jj - 1u : 0u];
      }
#pragma unroll
      for (int r = 0; r < EPL; ++r) {
        const uint32_t j = j0 + (uint32_t)r * WAVE + lane;
        if (j < k) {
          const uint32_t i = ei[r];
          if (i >= L) {
            bad = 1u;
            vo[j] = R{};
          } else {
            if (j > 0 && i <= ep[r]) bad = 1u;   // not ascending
            const float X = b[i];
            vo[j] = Elem<T>::down(X);
            b[i] = X - through<T>(X);
          }
        }
      }
    }
    if (a.blk && (bt0 != 0u || bt1 != k)) bad = 1u;
    if (bad) raise_error(KERR_BAD_INDEX);
    __builtin_amdgcn_wave_barrier();
    for (uint32_t q = lane; q * 4 < L; q += WAVE) {
      if (vec) {
        vstore<true>(reinterpret_cast<u32x4*>(es) + q, reinterpret_cast<const u32x4*>(b)[q]);
      } else {
        for (uint32_t c = q * 4; c < min(L, q * 4 + 4); ++c) es[c] = b[c];
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

hipError_t launch_gather(int dt, const GatherArgs& args, hipStream_t st) {
  GatherArgs a = args;
  void* params[] = {&a};
  const void* fn;
  uint64_t work;
  if (a.e && a.L <= SR_MAX) {
    // one wavefront per row
    fn = (dt == DT_F32) ? (const void*)k_gather_ef_row<float>
       : (dt == DT_BF16) ? (const void*)k_gather_ef_row<bf16_t> : (const void*)k_gather_ef_row<f16_t>;
    work = (a.n_seg + SR_WAVES - 1) / SR_WAVES;
  } else if (a.e) {
    fn = (dt == DT_F32) ? (const void*)k_gather_ef<float>
       : (dt == DT_BF16) ? (const void*)k_gather_ef<bf16_t> : (const void*)k_gather_ef<f16_t>;
    work = a.n_seg * ((a.L + SC_CH - 1) / SC_CH);
  } else {
    fn = (dt == DT_F32) ? (const void*)k_gather<float>
       : (dt == DT_BF16) ? (const void*)k_gather<bf16_t> : (const void*)k_gather<f16_t>;
    work = (a.n_seg * a.k + SC_NT - 1) / SC_NT;
  }
  const uint32_t grid = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(work, (uint64_t)device_cus() * 8));
  return hipLaunchKernel(fn, dim3(grid), dim3(SC_NT), params, 0, st);
}

TC_DEFINE_ERROR_READER(errors_scatter)

}  // namespace tc
