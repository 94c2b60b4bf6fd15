// tc_internal.hpp -- launch plans and launcher entry points shared by the
// C-ABI layer (tc_api.cpp) and the kernel translation units.  Not installed.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tc {

enum Dt : int { DT_F32 = 0, DT_BF16 = 1, DT_F16 = 2 };

inline size_t dt_size(int dt) { return dt == DT_F32 ? 4u : 2u; }

// How one segmented kernel is laid out on the device: NT threads per
// workgroup, VPT consecutive elements per thread, P workgroups per segment
// (a "group"), n_groups groups resident at once (grid = n_groups * P), each
// looping over segments group, group + n_groups, ...
struct SegPlan {
  int nt = 0;
  int vpt = 0;
  uint32_t P = 1;
  uint32_t n_groups = 0;
  uint32_t grid = 0;
  uint64_t capacity = 0;   // workgroups of this kernel the device holds at once
  uint64_t ws_words = 0;   // 32-bit words of zero-initialised workspace needed
  uint64_t ws_used = 0;    // of which this launch touches (its n_groups groups)
  bool lds = false;        // TopK: one workgroup per segment held in LDS (k_topk_lds)
};

// ------------------------------------------------------------------- TopK
enum SelKind : int { SEL_PLAIN = 0, SEL_EF = 1, SEL_AQSGD = 2, SEL_EFMIX = 3 };

struct TopkArgs {
  const void* x;         // PLAIN/EF: [n_seg][L] input; AQSGD: activations [n_seg][L]
  float* e;              // EF: [n_seg][L] residual (in-out)
  void* m;               // AQSGD: buffer [n_samples][L] (in-out)
  const int64_t* ids;    // AQSGD: [n_seg] sample ids (device)
  uint64_t n_samples;
  uint32_t* idx;         // [n_seg][k]
  void* val;             // [n_seg][k] in the input dtype
  uint32_t* blk;         // optional [n_seg][nblk + 1] block table
  uint64_t n_seg, L, k;
  uint32_t P;
  uint32_t* ws;
  // EFMIX: the error buffer's list (idx, val, blk above hold the input's)
  uint32_t* idx2;        // [n_seg][k2]
  void* val2;            // [n_seg][k2] in the input dtype
  uint32_t* blk2;        // optional block table of that list
  uint64_t k2;
};

constexpr uint64_t BLOCK_LEN = 4096;   // TC_BLOCK_LEN
__host__ __device__ constexpr uint64_t n_blocks(uint64_t L) { return (L + BLOCK_LEN - 1) / BLOCK_LEN; }

SegPlan plan_topk(int sel, int dt, uint64_t n_seg, uint64_t L);
// the LDS engine (one workgroup per segment of at most LDS_SEG_MAX elements)
// for any such length; EF-mixed always takes it
constexpr uint64_t LDS_SEG_MAX = 32768;
SegPlan plan_lds(int sel, int dt, uint64_t n_seg);
hipError_t launch_topk(int sel, int dt, const SegPlan& plan, const TopkArgs& a, hipStream_t st);

// ----------------------------------------------------------- quantization
struct QuantArgs {
  const void* x;         // [n_grp][G]
  float* e;              // EF residual [n_grp][G] or nullptr
  uint32_t* codes;       // [n_grp][wpg] words
  float* meta;           // [n_grp][2]
  uint64_t n_grp, G, wpg;
  uint32_t P;
  uint32_t* ws;
};

SegPlan plan_quant(int dt, uint32_t bits, bool ef, uint64_t n_grp, uint64_t G);
hipError_t launch_quant(int dt, int out_dt, uint32_t bits, bool ef, const SegPlan& plan,
                        const QuantArgs& a, hipStream_t st);

struct UnpackArgs {
  const uint32_t* codes;
  const float* meta;
  void* y;
  uint64_t n_grp, G, wpg;
};
hipError_t launch_unpack(int out_dt, uint32_t bits, const UnpackArgs& a, hipStream_t st);

// --------------------------------------------------------- receiver side
struct ScatterArgs {
  const uint32_t* idx;   // [n_seg][k]
  const uint32_t* blk;   // optional [n_seg][nblk + 1] block table
  const void* val;       // [n_seg][k] wire values (TopK)
  const uint32_t* codes; // TopK+quant: [n_seg][wpg] codes of the kept list
  const float* meta;     // TopK+quant: [n_seg][2]
  void* y;               // dense output [n_seg][L]
  void* m;               // AQ-SGD receiver buffer [n_samples][L]
  const int64_t* ids;
  uint64_t n_samples;
  uint64_t n_seg, L, k, wpg;
  // EF-mixed: the error buffer's list, added after the input's
  const uint32_t* idx2;  // [n_seg][k2]
  const uint32_t* blk2;  // optional block table of that list
  const void* val2;      // [n_seg][k2] wire values
  uint64_t k2;
};
hipError_t launch_topk_decompress(int wire, int out_dt, const ScatterArgs& a, hipStream_t st);
hipError_t launch_efmix_recv(int wire, int out_dt, const ScatterArgs& a, hipStream_t st);

// EF-mixed residual after both selections (the sender's second kernel)
struct EfmixResidArgs {
  const void* x;         // [n_seg][L] input
  float* e;              // [n_seg][L] residual (in-out)
  const uint32_t* idx;   // the input's list [n_seg][k]
  const uint32_t* blk;   // its block table or nullptr
  const uint32_t* idx2;  // the buffer's list [n_seg][k2]
  const uint32_t* blk2;  // its block table or nullptr
  uint64_t n_seg, L, k, k2;
};
hipError_t launch_efmix_resid(int dt, const EfmixResidArgs& a, hipStream_t st);

// TopK at given indices (another tensor's TopK payload), optionally inside
// error feedback
struct GatherArgs {
  const uint32_t* idx;   // [n_seg][k], ascending per segment
  const uint32_t* blk;   // optional block table of that payload
  const void* x;         // [n_seg][L]
  float* e;              // EF residual [n_seg][L] (in-out) or nullptr
  void* val;             // [n_seg][k] in x's dtype
  uint64_t n_seg, L, k;
};
hipError_t launch_gather(int dt, const GatherArgs& a, hipStream_t st);
hipError_t launch_aqsgd_recv(int dt, const ScatterArgs& a, hipStream_t st);

// ------------------------------------------------ segments too long to hold
// TopK over one segment with a chain of kernels (a sampled band, candidate
// or whole-segment radix passes, per-tile counts and their offsets, an emit
// pass that writes each tile's kept entries at its offset, the kept-list
// quantizer)
struct GlobalArgs {
  const void* x;         // [L] input
  float* e;              // [L] residual (in-out) or nullptr
  uint32_t* idx;         // [k]
  void* val;             // [k] wire values (plain TopK) or nullptr
  uint32_t* codes;       // quantized kept list: [wpg] words
  float* meta;           // quantized kept list: [2]
  uint32_t* blk;         // optional [n_blocks(L) + 1]
  uint64_t L, k, wpg, n_tiles;
  uint32_t* state;       // workspace pieces (global_ws_carve)
  uint32_t* hist;
  uint32_t* tiles;       // 4 words per tile
  uint32_t* wgs;         // tile-count workgroup totals / prefixes
  uint32_t* cand;        // candidate sub-lists: binary32 bits of the values in the band
  uint64_t cand_cap;     // all sub-lists together
  uint32_t bits;         // quantized kept list: b (0: values)
  uint32_t sample_stride;
  uint32_t n_sub;        // candidate sub-lists (<= 8, <= the chain's grid)
  uint32_t tpw;          // tiles per tile-count workgroup
};
uint64_t global_ws_words(uint64_t L);
void global_ws_carve(uint32_t* ws, uint64_t L, GlobalArgs& a);
hipError_t launch_global(int dt, bool ef, uint32_t qbits, const GlobalArgs& a, hipStream_t st);

// ------------------------------------ preconditions (debug library only)
// Bits the check kernels of k_check.hip report; each call synchronizes the
// stream and returns the bits found (and clears them).
enum : uint32_t { CHK_NONFINITE = 1u, CHK_RANGE = 2u };
hipError_t check_values(int dt, const void* x, const float* e, uint64_t n, hipStream_t st, uint32_t* flags);
hipError_t check_aqsgd(int dt, const void* a, const void* m, const int64_t* ids, uint64_t n_ids, uint64_t L,
                       uint64_t n_samples, hipStream_t st, uint32_t* flags);

// sticky kernel error bits of each kernel translation unit
hipError_t errors_topk(uint32_t* bits, bool clear);
hipError_t errors_quant(uint32_t* bits, bool clear);
hipError_t errors_scatter(uint32_t* bits, bool clear);
hipError_t errors_global(uint32_t* bits, bool clear);
// the same words set from the host (tests of the recovery path)
hipError_t errors_topk_raise(uint32_t bits);
hipError_t errors_quant_raise(uint32_t bits);
hipError_t errors_scatter_raise(uint32_t bits);
hipError_t errors_global_raise(uint32_t bits);

// device properties (cached per device)
int device_cus();

// ---- library-owned scratch of the allocation-free entry point (k_scratch.hip)
constexpr uint64_t NOALLOC_SCRATCH_BYTES = 4ull << 20;    // TC_NOALLOC_SCRATCH_BYTES
hipError_t noalloc_scratch(void** ptr, hipStream_t st);
hipError_t noalloc_scratch_reset();

}  // namespace tc
