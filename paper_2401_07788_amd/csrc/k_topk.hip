// k_topk.hip -- the sender side of TopK (Sec. 2.3), with error feedback
// (Sec. 2.4) or AQ-SGD (Sec. 2.5) fused around it.
//
// One kernel body, three producers / epilogues:
//   PLAIN : v = x                                  -> payload
//   EF    : v = x + e                              -> payload, e <- v - r
//           r = what the receiver gets: wire(v) at kept entries, +0 elsewhere
//   AQSGD : v = a - m[id]                          -> payload, m[id][kept] += wire(v)
// The segment (a sample, a token row, a whole tensor) stays in registers for
// the whole kernel: inputs are read once, the selection passes work on
// registers and LDS, and the outputs are written once.
#include <algorithm>
#include <type_traits>

#include "tc_internal.hpp"
#include "tc_select.hpp"

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

struct RowShared {
  uint32_t scratch[2];
};

// LDS of the several-workgroup layout: the selection histogram, and after
// the selection the workgroup's payload entries, staged so that they leave
// in index order with coalesced stores
template <int NT, int VPT, typename R>
union BigShared {
  SelShared<NT> sel;
  struct {
    uint32_t idx[NT * VPT];
    R val[NT * VPT];
  } st;
};

template <typename InT, int SEL, int VPT, int NT>
__global__ __launch_bounds__(NT) void k_topk_seg(TopkArgs a) {
  using R = typename Elem<InT>::raw;
  constexpr bool BIG = NT > WAVE;
  using Sh = std::conditional_t<BIG, BigShared<NT, VPT, R>, RowShared>;
  __shared__ Sh sh;
  constexpr uint64_t CH = (uint64_t)NT * VPT;

  const uint32_t P = a.P;
  uint32_t group, part;
  map_wg(blockIdx.x, gridDim.x, P, group, part);
  const uint32_t n_groups = gridDim.x / P;
  GroupMem gm{};
  if constexpr (BIG) {
    if (P > 1) gm = group_mem(a.ws, group, P);
  }
  bool exited = false;

  for (uint64_t seg = group; seg < a.n_seg; seg += n_groups) {
    const uint64_t c0 = (uint64_t)part * CH + (uint64_t)threadIdx.x * VPT;
    const int nv = (int)min((uint64_t)VPT, sat_sub(a.L, c0));

    // ---- producer: the vector to compress, in binary32
    float v[VPT];
    R mr[VPT];                 // AQSGD: the buffer row, kept for the update
    uint64_t mrow = 0;
    if constexpr (SEL == SEL_AQSGD) {
      const int64_t id = a.ids[seg];
      if (id < 0 || (uint64_t)id >= a.n_samples) {
        if (threadIdx.x == 0 && part == 0) raise_error(KERR_BAD_ID);
        continue;              // every workgroup of the group skips alike
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

    // ---- selection
    SelResult sr;
    Placement pl;
    if constexpr (BIG) {
      if (a.k == 0) { sr.T = 0xFFFFFFFFu; sr.r = 0; sr.gt_before = 0; sr.eq_before = 0; }
      else sr = radix_select<NT, VPT>(key, nv, (uint32_t)a.k, P, part, gm, sh.sel);
      pl = place<NT, VPT>(key, nv, sr, sh.sel.scratch);
      // the group's slots have been read: count out now, before the writes
      if (P > 1 && seg + n_groups >= a.n_seg) {
        group_exit<NT>(gm.bar, P, gm.slots, slot_words(P));
        exited = true;
      }
    } else {
      if (a.k == 0) { sr.T = 0xFFFFFFFFu; sr.r = 0; sr.gt_before = 0; sr.eq_before = 0; }
      else sr = bitwise_select<VPT>(key, nv, (uint32_t)a.k);
      pl = place<NT, VPT>(key, nv, sr, sh.scratch);
    }

    // ---- payload + epilogue
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
          if constexpr (BIG) {
            const uint32_t li = pos - pl.wg_first;     // slot inside the workgroup's run
            if (li < CH) { sh.st.idx[li] = (uint32_t)(c0 + i); sh.st.val[li] = w; }
            else raise_error(KERR_INTERNAL);
          } else {
            if (pos < a.k) { idx[pos] = (uint32_t)(c0 + i); val[pos] = w; }
            else raise_error(KERR_INTERNAL);
          }
          ++pos;
          if constexpr (SEL == SEL_AQSGD) mr[i] = Elem<InT>::down(Elem<InT>::up(mr[i]) + Elem<InT>::up(w));
        }
      }
      if constexpr (SEL == SEL_EF) eo[i] = v[i] - (kept ? through<InT>(v[i]) : 0.0f);
    }
    if constexpr (SEL == SEL_EF) {
      if (nv > 0) store_run_partial<float, VPT, false>(a.e + seg * a.L + c0, nv, eo);
    }
    if constexpr (SEL == SEL_AQSGD) {
      if (nv > 0 && a.k > 0) store_run_partial<R, VPT, false>((R*)a.m + mrow + c0, nv, mr);
    }
    if constexpr (BIG) {
      // the workgroup's run of the payload, in index order, coalesced
      __syncthreads();
      const uint32_t cnt = min(pl.wg_count, (uint32_t)CH);
      if (pl.wg_first + cnt > a.k) { if (threadIdx.x == 0) raise_error(KERR_INTERNAL); }
      else {
        copy_lds_to_global<NT>(idx + pl.wg_first, sh.st.idx, cnt);
        copy_lds_to_global<NT>(val + pl.wg_first, sh.st.val, cnt);
      }
      // block table: kept entries below each block boundary this workgroup covers,
      // found by a lower bound in the staged (ascending) run
      if (a.blk) {
        uint32_t* bt = a.blk + seg * (n_blocks(a.L) + 1);
        const uint64_t w0 = (uint64_t)part * CH, w1 = min(a.L, w0 + CH);
        for (uint64_t b = (w0 + BLOCK_LEN - 1) / BLOCK_LEN + threadIdx.x; b * BLOCK_LEN < w1; b += NT) {
          const uint64_t B = b * BLOCK_LEN;
          uint32_t lo = 0, hi = cnt;
          while (lo < hi) {
            const uint32_t mid = (lo + hi) >> 1;
            if (sh.st.idx[mid] < B) lo = mid + 1; else hi = mid;
          }
          bt[b] = pl.wg_first + lo;
        }
        if (part == 0 && threadIdx.x == 0) bt[n_blocks(a.L)] = (uint32_t)a.k;
      }
      __syncthreads();
    } else {
      if (a.blk && threadIdx.x == 0) {
        // a wavefront segment is shorter than one block
        uint32_t* bt = a.blk + seg * (n_blocks(a.L) + 1);
        bt[0] = 0;
        bt[n_blocks(a.L)] = (uint32_t)a.k;
      }
    }
  }
  if constexpr (BIG) {
    if (P > 1 && !exited) group_exit<NT>(gm.bar, P, gm.slots, slot_words(P));
  }
}

// ------------------------------------------------------------------ plans
namespace {

constexpr int BIG_NT = 512;
constexpr int ROW_NT = 64;
constexpr uint64_t ROW_MAX = (uint64_t)ROW_NT * 32;   // longest segment one wavefront holds
static_assert(ROW_MAX <= BLOCK_LEN, "a wavefront segment fits in one block of the block table");

template <typename InT, int SEL>
const void* kernel_ptr(int nt, int vpt) {
  if (nt == ROW_NT) {
    switch (vpt) {
      case 4: return (const void*)k_topk_seg<InT, SEL, 4, ROW_NT>;
      case 8: return (const void*)k_topk_seg<InT, SEL, 8, ROW_NT>;
      case 12: return (const void*)k_topk_seg<InT, SEL, 12, ROW_NT>;
      case 16: return (const void*)k_topk_seg<InT, SEL, 16, ROW_NT>;
      case 24: return (const void*)k_topk_seg<InT, SEL, 24, ROW_NT>;
      case 32: return (const void*)k_topk_seg<InT, SEL, 32, ROW_NT>;
    }
  } else {
    switch (vpt) {
      case 4: return (const void*)k_topk_seg<InT, SEL, 4, BIG_NT>;
      case 8: return (const void*)k_topk_seg<InT, SEL, 8, BIG_NT>;
      case 16: return (const void*)k_topk_seg<InT, SEL, 16, BIG_NT>;
      case 24: return (const void*)k_topk_seg<InT, SEL, 24, BIG_NT>;
    }
  }
  return nullptr;
}

template <int SEL>
const void* kernel_ptr_dt(int dt, int nt, int vpt) {
  if (dt == DT_F32) return kernel_ptr<float, SEL>(nt, vpt);
  if (dt == DT_BF16) return kernel_ptr<bf16_t, SEL>(nt, vpt);
  return kernel_ptr<f16_t, SEL>(nt, vpt);
}

const void* pick(int sel, int dt, int nt, int vpt) {
  if (sel == SEL_PLAIN) return kernel_ptr_dt<SEL_PLAIN>(dt, nt, vpt);
  if (sel == SEL_EF) return kernel_ptr_dt<SEL_EF>(dt, nt, vpt);
  return kernel_ptr_dt<SEL_AQSGD>(dt, nt, vpt);
}

int occupancy(const void* fn, int nt) {
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, fn, nt, 0) != hipSuccess || blocks < 1) blocks = 1;
  return blocks;
}

}  // namespace

SegPlan plan_topk(int sel, int dt, uint64_t n_seg, uint64_t L) {
  SegPlan p;
  const uint32_t cus = (uint32_t)device_cus();
  if (L <= ROW_MAX) {
    // one wavefront per segment: the smallest run length that covers L
    static const int vpts[] = {4, 8, 12, 16, 24, 32};
    p.nt = ROW_NT;
    for (int v : vpts) { p.vpt = v; if ((uint64_t)ROW_NT * v >= L) break; }
    p.P = 1;
    const uint64_t cap = (uint64_t)occupancy(pick(sel, dt, p.nt, p.vpt), p.nt) * cus;
    p.capacity = cap;
    p.n_groups = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(n_seg, cap));
    p.grid = p.n_groups;
    p.ws_words = 0;
    return p;
  }
  // several workgroups per segment: the longest run per thread that still
  // gives every compute unit a workgroup, else the shortest run
  static const int vpts[] = {24, 16, 8, 4};
  p.nt = BIG_NT;
  p.vpt = 4;
  for (int v : vpts) {
    const uint64_t P = (L + (uint64_t)BIG_NT * v - 1) / ((uint64_t)BIG_NT * v);
    if (n_seg * P >= cus) { p.vpt = v; break; }
  }
  const uint64_t CH = (uint64_t)BIG_NT * p.vpt;
  p.P = (uint32_t)((L + CH - 1) / CH);
  const uint64_t cap = (uint64_t)occupancy(pick(sel, dt, p.nt, p.vpt), p.nt) * cus;
  p.capacity = cap;
  uint64_t groups = std::min<uint64_t>(n_seg, std::max<uint64_t>(1, cap / p.P));
  if (p.P > 1 && groups >= 8) groups -= groups % 8;
  p.n_groups = (uint32_t)groups;
  p.grid = (uint32_t)(groups * p.P);
  // the workspace is sized for the most groups any instance could keep
  // resident (4 workgroups of 512 threads per compute unit), so that one size
  // serves every selection kind of the same layout
  const uint64_t ws_groups = std::min<uint64_t>(n_seg, std::max<uint64_t>(1, (uint64_t)cus * 4 / p.P));
  p.ws_words = (p.P > 1) ? ws_groups * group_mem_words(p.P) : 0;
  return p;
}

hipError_t launch_topk(int sel, int dt, const SegPlan& plan, const TopkArgs& args, hipStream_t st) {
  const void* fn = pick(sel, dt, plan.nt, plan.vpt);
  if (!fn) return hipErrorInvalidValue;
  TopkArgs a = args;
  a.P = plan.P;
  void* params[] = {&a};
  return hipLaunchKernel(fn, dim3(plan.grid), dim3(plan.nt), params, 0, st);
}

TC_DEFINE_ERROR_READER(errors_topk)

}  // namespace tc
