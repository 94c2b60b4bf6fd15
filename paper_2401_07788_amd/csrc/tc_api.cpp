// tc_api.cpp -- the C ABI declared in include/tc.h: argument validation,
// launch planning and status reporting.  No device memory is allocated here.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <vector>

#include "../../include/tc.h"
#include "tc_internal.hpp"

#define TC_API extern "C" __attribute__((visibility("default")))

static_assert(TC_NOALLOC_SCRATCH_BYTES == tc::NOALLOC_SCRATCH_BYTES, "one scratch size");

namespace tc {

int device_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

}  // namespace tc

namespace {

thread_local char g_err[512] = "";

tc_status fail(tc_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

tc_status hip_fail(hipError_t e, const char* what) {
  return fail(TC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool dt_ok(int dt) { return dt == TC_F32 || dt == TC_BF16 || dt == TC_F16; }
bool bits_ok(uint32_t b) { return (b >= 1 && b <= 8) || b == 32; }

// common codec checks; `need_k` for TopK-based kinds
tc_status check_codec(const tc_codec* c, int kind_mask) {
  if (!c) return fail(TC_ERR_NULL, "codec is NULL");
  if (c->kind < TC_TOPK || c->kind > TC_TOPK_QUANT) return fail(TC_ERR_ARG, "codec.kind %d", c->kind);
  if (c->reserved != 0) return fail(TC_ERR_ARG, "codec.reserved must be 0");
  if (!((1 << c->kind) & kind_mask)) return fail(TC_ERR_ARG, "codec.kind %d not valid for this call", c->kind);
  if (c->seg_len >= (1ull << 32)) return fail(TC_ERR_ARG, "seg_len %llu must be < 2^32", (unsigned long long)c->seg_len);
  if (c->n_seg != 0 && c->seg_len != 0 && c->n_seg > UINT64_MAX / c->seg_len)
    return fail(TC_ERR_ARG, "n_seg * seg_len overflows");
  if (c->kind == TC_TOPK || c->kind == TC_TOPK_QUANT) {
    if (c->k > c->seg_len) return fail(TC_ERR_ARG, "k %llu > seg_len %llu", (unsigned long long)c->k,
                                       (unsigned long long)c->seg_len);
  }
  if (c->kind == TC_QUANT || c->kind == TC_TOPK_QUANT) {
    if (!bits_ok(c->bits)) return fail(TC_ERR_ARG, "bits %u not in 1..8 or 32", c->bits);
  }
  return TC_OK;
}

tc_status check_ws(const tc::SegPlan& p, const void* ws, size_t ws_bytes) {
  const size_t need = (size_t)p.ws_words * 4u;
  if (need == 0) return TC_OK;
  if (!ws) return fail(TC_ERR_WORKSPACE, "workspace of %zu bytes required", need);
  if (ws_bytes < need) return fail(TC_ERR_WORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, need);
  if (((uintptr_t)ws & 7u) != 0) return fail(TC_ERR_ALIGN, "workspace must be 8-byte aligned");
  return TC_OK;
}

// a segment spread over more workgroups than the device holds at once cannot
// use the register-resident kernels
tc_status check_resident(const tc::SegPlan& p) {
  if (p.n_groups == 0 || p.P > p.capacity)
    return fail(TC_ERR_ARG, "a segment needs %u workgroups at once, the device holds %llu", p.P,
                (unsigned long long)p.capacity);
  return TC_OK;
}

#ifdef TC_DEBUG
// ---- precondition checks of the debug library (see "Preconditions" in tc.h)
struct Span {
  const void* p;
  uint64_t bytes;
  const char* name;
};

// no two of a call's buffers overlap
tc_status check_disjoint(std::initializer_list<Span> spans) {
  for (auto i = spans.begin(); i != spans.end(); ++i)
    for (auto j = i + 1; j != spans.end(); ++j) {
      if (!i->p || !j->p || i->bytes == 0 || j->bytes == 0) continue;
      const uintptr_t a0 = (uintptr_t)i->p, b0 = (uintptr_t)j->p;
      if (a0 < b0 + j->bytes && b0 < a0 + i->bytes)
        return fail(TC_ERR_PRECONDITION, "%s and %s overlap", i->name, j->name);
    }
  return TC_OK;
}

// AQ-SGD: no sample id twice in one call (read back through the stream)
tc_status check_ids_distinct(const int64_t* ids, uint64_t n_ids, void* stream) {
  if (n_ids < 2) return TC_OK;
  std::vector<int64_t> h(n_ids);
  hipError_t e = hipMemcpyAsync(h.data(), ids, n_ids * sizeof(int64_t), hipMemcpyDeviceToHost, (hipStream_t)stream);
  if (e == hipSuccess) e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "reading the ids for the precondition check");
  std::sort(h.begin(), h.end());
  for (size_t i = 1; i < h.size(); ++i)
    if (h[i] == h[i - 1]) return fail(TC_ERR_PRECONDITION, "sample id %lld appears twice in one call", (long long)h[i]);
  return TC_OK;
}

tc_status check_flags(hipError_t e, uint32_t flags, const char* what) {
  if (e != hipSuccess) return hip_fail(e, what);
  if (flags & tc::CHK_NONFINITE) return fail(TC_ERR_PRECONDITION, "%s: a value is not finite", what);
  if (flags & tc::CHK_RANGE)
    return fail(TC_ERR_PRECONDITION, "%s: a value is too large for its range or update to stay finite", what);
  return TC_OK;
}

tc_status check_values(int dt, const void* x, const float* e, uint64_t n, void* stream) {
  uint32_t flags = 0;
  const hipError_t he = tc::check_values(dt, x, e, n, (hipStream_t)stream, &flags);
  return check_flags(he, flags, "input check");
}

#define TC_PRECONDITION(expr)            \
  do {                                   \
    const tc_status s_ = (expr);         \
    if (s_ != TC_OK) return s_;          \
  } while (0)
#else
#define TC_PRECONDITION(expr) \
  do {                        \
  } while (0)
#endif

uint64_t bytes_of(uint64_t n, int dt) { return n * tc::dt_size(dt); }

tc_status check_aqsgd_args(const tc_codec* c, uint64_t n_samples, uint32_t n_ids) {
  tc_status s = check_codec(c, 1 << TC_TOPK);
  if (s != TC_OK) return s;
  if (c->n_seg != n_ids) return fail(TC_ERR_ARG, "codec.n_seg %llu != n_ids %u", (unsigned long long)c->n_seg, n_ids);
  if (n_ids > 0 && n_samples == 0) return fail(TC_ERR_ARG, "n_samples is 0");
  if (c->seg_len != 0 && n_samples > UINT64_MAX / c->seg_len) return fail(TC_ERR_ARG, "n_samples * seg_len overflows");
  return TC_OK;
}

// TopK of segments too long to keep on chip, one segment after the other
// (see k_global.hip); qbits != 0 quantizes the kept list (needs e)
tc_status global_topk(uint32_t qbits, const tc_codec* c, const void* x, int dt, float* e, const tc_payload* out,
                      void* ws, size_t ws_bytes, void* stream) {
  const uint64_t L = c->seg_len, k = c->k;
  if (L >= (1ull << 31)) return fail(TC_ERR_ARG, "seg_len %llu must be < 2^31 for a segment this long",
                                     (unsigned long long)L);
  const size_t need = (size_t)tc::global_ws_words(L) * 4u;
  if (!ws) return fail(TC_ERR_WORKSPACE, "workspace of %zu bytes required", need);
  if (ws_bytes < need) return fail(TC_ERR_WORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, need);
  if (((uintptr_t)ws & 7u) != 0) return fail(TC_ERR_ALIGN, "workspace must be 8-byte aligned");
  const uint64_t gb = qbits ? tc_quant_group_bytes(k, qbits) : 0;
  const uint64_t nb = tc::n_blocks(L) + 1;
  for (uint64_t s = 0; s < c->n_seg; ++s) {
    tc::GlobalArgs a{};
    a.x = (const char*)x + s * L * tc::dt_size(dt);
    a.e = e ? e + s * L : nullptr;
    a.idx = out->idx ? out->idx + s * k : nullptr;
    a.val = (!qbits && out->val) ? (char*)out->val + s * k * tc::dt_size(dt) : nullptr;
    a.codes = qbits ? (uint32_t*)(out->codes + s * gb) : nullptr;
    a.meta = qbits ? out->meta + 2 * s : nullptr;
    a.blk = out->blk ? out->blk + s * nb : nullptr;
    a.L = L;
    a.k = k;
    a.wpg = gb / 4u;
    tc::global_ws_carve((uint32_t*)ws, L, a);
    hipError_t he = tc::launch_global(dt, e != nullptr, qbits, a, (hipStream_t)stream);
    if (he != hipSuccess) return hip_fail(he, "global topk launch");
  }
  return TC_OK;
}

// noalloc: the workspace is the library's own scratch (ws, ws_bytes unused)
tc_status topk_common(int sel, const tc_codec* c, const void* x, int dt, float* e, void* m, uint64_t n_samples,
                      const int64_t* ids, const tc_payload* out, void* ws, size_t ws_bytes, void* stream,
                      bool noalloc = false) {
  if (!dt_ok(dt)) return fail(TC_ERR_DTYPE, "dtype %d", dt);
  if (c->wire != dt) return fail(TC_ERR_DTYPE, "wire dtype %d must equal the input dtype %d", c->wire, dt);
  if (!out) return fail(TC_ERR_NULL, "payload is NULL");
  const uint64_t n = c->n_seg * c->seg_len;
  if (n == 0) return TC_OK;
  if (!x) return fail(TC_ERR_NULL, "input is NULL");
  if (sel == tc::SEL_EF && !e) return fail(TC_ERR_NULL, "error buffer is NULL");
  if (sel == tc::SEL_AQSGD && (!m || !ids)) return fail(TC_ERR_NULL, "buffer or ids is NULL");
  if (c->k > 0 && (!out->idx || !out->val)) return fail(TC_ERR_NULL, "payload idx/val is NULL");
  const uint64_t nb = tc::n_blocks(c->seg_len) + 1;
  TC_PRECONDITION(check_disjoint({{x, bytes_of(n, dt), "input"},
                                  {e, 4 * n, "e"},
                                  {m, bytes_of(n_samples * c->seg_len, dt), "m"},
                                  {ids, 8 * c->n_seg, "ids"},
                                  {out->idx, 4 * c->n_seg * c->k, "payload idx"},
                                  {out->val, bytes_of(c->n_seg * c->k, dt), "payload val"},
                                  {out->blk, 4 * c->n_seg * nb, "payload blk"},
                                  {ws, ws_bytes, "workspace"}}));
  if (sel == tc::SEL_AQSGD) {
    TC_PRECONDITION(check_ids_distinct(ids, c->n_seg, stream));
#ifdef TC_DEBUG
    uint32_t flags = 0;
    const hipError_t he = tc::check_aqsgd(dt, x, m, ids, c->n_seg, c->seg_len, n_samples, (hipStream_t)stream, &flags);
    TC_PRECONDITION(check_flags(he, flags, "AQ-SGD input check"));
#endif
  } else {
    TC_PRECONDITION(check_values(dt, x, e, n, stream));
  }
  // k == 0: an empty payload (and, for AQ-SGD, an unchanged buffer); only a
  // requested block table still has to be written
  if (c->k == 0 && !out->blk && (sel == tc::SEL_PLAIN || sel == tc::SEL_AQSGD)) return TC_OK;
  const tc::SegPlan p = tc::plan_topk(sel, dt, c->n_seg, c->seg_len);
  tc_status s = check_resident(p);
  if (s != TC_OK) {
    if (sel == tc::SEL_AQSGD) return s;
    g_err[0] = 0;
    return global_topk(0, c, x, dt, e, out, ws, ws_bytes, stream);   // too long for one resident group
  }
  if (noalloc) {
    const uint64_t need = p.ws_used * 4u;
    if (need > tc::NOALLOC_SCRATCH_BYTES)
      return fail(TC_ERR_WORKSPACE, "this shape needs %llu bytes of scratch, the allocation-free entry point holds %llu",
                  (unsigned long long)need, (unsigned long long)tc::NOALLOC_SCRATCH_BYTES);
    ws = nullptr;
    ws_bytes = 0;
    if (need > 0) {
      const hipError_t he = tc::noalloc_scratch(&ws, (hipStream_t)stream);
      if (he != hipSuccess) return hip_fail(he, "scratch set-up");
      ws_bytes = tc::NOALLOC_SCRATCH_BYTES;
    }
  } else {
    s = check_ws(p, ws, ws_bytes);
    if (s != TC_OK) return s;
  }
  tc::TopkArgs a{};
  a.x = x;
  a.e = e;
  a.m = m;
  a.ids = ids;
  a.n_samples = n_samples;
  a.idx = out->idx;
  a.val = out->val;
  a.blk = out->blk;
  a.n_seg = c->n_seg;
  a.L = c->seg_len;
  a.k = c->k;
  a.ws = (uint32_t*)ws;
  hipError_t he = tc::launch_topk(sel, dt, p, a, (hipStream_t)stream);
  if (he != hipSuccess) return hip_fail(he, "topk launch");
  return TC_OK;
}

tc_status quant_common(bool ef, const tc_codec* c, const void* x, int dt, float* e, const tc_payload* out,
                       void* ws, size_t ws_bytes, void* stream) {
  if (!dt_ok(dt)) return fail(TC_ERR_DTYPE, "dtype %d", dt);
  if (!out) return fail(TC_ERR_NULL, "payload is NULL");
  const uint64_t n = c->n_seg * c->seg_len;
  if (n == 0) return TC_OK;
  if (!x) return fail(TC_ERR_NULL, "input is NULL");
  if (ef && !e) return fail(TC_ERR_NULL, "error buffer is NULL");
  if (!out->codes || !out->meta) return fail(TC_ERR_NULL, "payload codes/meta is NULL");
  if (((uintptr_t)out->codes & 3u) != 0) return fail(TC_ERR_ALIGN, "codes must be 4-byte aligned");
  TC_PRECONDITION(check_disjoint({{x, bytes_of(n, dt), "input"},
                                  {e, 4 * n, "e"},
                                  {out->codes, c->n_seg * tc_quant_group_bytes(c->seg_len, c->bits), "codes"},
                                  {out->meta, 8 * c->n_seg, "meta"},
                                  {ws, ws_bytes, "workspace"}}));
  TC_PRECONDITION(check_values(dt, x, e, n, stream));
  const tc::SegPlan p = tc::plan_quant(dt, c->bits, ef, c->n_seg, c->seg_len);
  tc_status s = check_resident(p);
  if (s != TC_OK) return s;
  s = check_ws(p, ws, ws_bytes);
  if (s != TC_OK) return s;
  tc::QuantArgs a{};
  a.x = x;
  a.e = e;
  a.codes = (uint32_t*)out->codes;
  a.meta = out->meta;
  a.n_grp = c->n_seg;
  a.G = c->seg_len;
  a.wpg = tc_quant_group_bytes(c->seg_len, c->bits) / 4u;
  a.ws = (uint32_t*)ws;
  hipError_t he = tc::launch_quant(dt, dt, c->bits, ef, p, a, (hipStream_t)stream);
  if (he != hipSuccess) return hip_fail(he, "quant launch");
  return TC_OK;
}

}  // namespace

TC_API uint64_t tc_topk_count(uint64_t seg_len, uint32_t num, uint32_t den) {
  if (den == 0) return 0;
  const unsigned __int128 p = (unsigned __int128)seg_len * num + (den - 1u);
  return (uint64_t)(p / den);
}

TC_API uint64_t tc_quant_group_bytes(uint64_t grp_len, uint32_t bits) {
  if (bits == 32) return 4u * grp_len;
  if (bits < 1 || bits > 8) return 0;
  return 4u * ((grp_len * bits + 31u) / 32u);
}

TC_API tc_status tc_workspace_bytes(const tc_codec* c, size_t* bytes) {
  if (!bytes) return fail(TC_ERR_NULL, "bytes is NULL");
  *bytes = 0;
  tc_status s = check_codec(c, (1 << TC_TOPK) | (1 << TC_QUANT) | (1 << TC_TOPK_QUANT));
  if (s != TC_OK) return s;
  if (c->n_seg * c->seg_len == 0) return TC_OK;
  uint64_t words = 0;
  const int dt = dt_ok(c->wire) ? c->wire : TC_F32;
  if (c->kind == TC_TOPK) {
    // enough for every sender kind of this shape (the plans of EF and
    // AQ-SGD differ where a plan has to fit a resident group); a segment too
    // long for them takes the global chain
    for (int sel : {tc::SEL_EF, tc::SEL_AQSGD}) {
      const tc::SegPlan p = tc::plan_topk(sel, dt, c->n_seg, c->seg_len);
      words = std::max<uint64_t>(words, (p.n_groups == 0 || p.P > p.capacity) ? tc::global_ws_words(c->seg_len)
                                                                              : p.ws_words);
    }
  } else if (c->kind == TC_QUANT) {
    words = std::max(tc::plan_quant(dt, c->bits, true, c->n_seg, c->seg_len).ws_words,
                     tc::plan_quant(dt, c->bits, false, c->n_seg, c->seg_len).ws_words);
  } else {
    words = tc::global_ws_words(c->seg_len);
  }
  *bytes = (size_t)words * 4u;
  return TC_OK;
}

TC_API void tc_efmix_counts(uint64_t k, uint64_t* k_x, uint64_t* k_e) {
  // reading E5: the input's list takes the odd entry
  if (k_x) *k_x = k - k / 2;
  if (k_e) *k_e = k / 2;
}

TC_API const char* tc_status_str(int s) {
  switch (s) {
    case TC_OK: return "ok";
    case TC_ERR_NULL: return "null pointer";
    case TC_ERR_ARG: return "invalid argument";
    case TC_ERR_DTYPE: return "unsupported dtype";
    case TC_ERR_WORKSPACE: return "workspace missing or too small";
    case TC_ERR_HIP: return "HIP runtime error";
    case TC_ERR_PRECONDITION: return "precondition violated (debug library)";
    case TC_ERR_ALIGN: return "misaligned buffer";
  }
  return "unknown status";
}

TC_API const char* tc_last_error(void) { return g_err; }

TC_API tc_status tc_device_errors(uint32_t* bits, int clear) {
  if (!bits) return fail(TC_ERR_NULL, "bits is NULL");
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
  uint32_t a = 0, b = 0, d = 0;
  if ((e = tc::errors_topk(&a, clear != 0)) != hipSuccess) return hip_fail(e, "error word (topk)");
  if ((e = tc::errors_quant(&b, clear != 0)) != hipSuccess) return hip_fail(e, "error word (quant)");
  if ((e = tc::errors_scatter(&d, clear != 0)) != hipSuccess) return hip_fail(e, "error word (scatter)");
  uint32_t g = 0;
  if ((e = tc::errors_global(&g, clear != 0)) != hipSuccess) return hip_fail(e, "error word (global)");
  *bits = a | b | d | g;
  // a wait that gave up leaves the allocation-free entry point's scratch dirty
  if (clear && (*bits & TC_KERR_TIMEOUT) && (e = tc::noalloc_scratch_reset()) != hipSuccess)
    return hip_fail(e, "clearing the scratch");
  return TC_OK;
}

TC_API tc_status tc_raise_device_errors(uint32_t bits) {
  if (bits & ~(uint32_t)(TC_KERR_TIMEOUT | TC_KERR_BAD_ID | TC_KERR_BAD_INDEX | TC_KERR_INTERNAL))
    return fail(TC_ERR_ARG, "bits %#x: unknown kernel error bits", bits);
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
  if ((e = tc::errors_topk_raise(bits)) != hipSuccess) return hip_fail(e, "error word (topk)");
  if ((e = tc::errors_quant_raise(bits)) != hipSuccess) return hip_fail(e, "error word (quant)");
  if ((e = tc::errors_scatter_raise(bits)) != hipSuccess) return hip_fail(e, "error word (scatter)");
  if ((e = tc::errors_global_raise(bits)) != hipSuccess) return hip_fail(e, "error word (global)");
  return TC_OK;
}

TC_API tc_status tc_topk_compress(const tc_codec* c, const void* x, int dt, const tc_payload* out, void* ws,
                                  size_t ws_bytes, void* stream) {
  tc_status s = check_codec(c, 1 << TC_TOPK);
  if (s != TC_OK) return s;
  return topk_common(tc::SEL_PLAIN, c, x, dt, nullptr, nullptr, 0, nullptr, out, ws, ws_bytes, stream);
}

TC_API tc_status tc_topk_decompress(const tc_codec* c, const tc_payload* in, void* y, int out_dt, void* stream) {
  tc_status s = check_codec(c, (1 << TC_TOPK) | (1 << TC_TOPK_QUANT));
  if (s != TC_OK) return s;
  if (!dt_ok(out_dt)) return fail(TC_ERR_DTYPE, "out dtype %d", out_dt);
  if (!in) return fail(TC_ERR_NULL, "payload is NULL");
  if (c->n_seg * c->seg_len == 0) return TC_OK;
  if (!y) return fail(TC_ERR_NULL, "output is NULL");
  if (c->k > 0 && !in->idx) return fail(TC_ERR_NULL, "payload idx is NULL");
  int wire;
  if (c->kind == TC_TOPK) {
    if (!dt_ok(c->wire)) return fail(TC_ERR_DTYPE, "wire dtype %d", c->wire);
    if (c->k > 0 && !in->val) return fail(TC_ERR_NULL, "payload val is NULL");
    wire = c->wire;
  } else {
    if (c->k > 0 && (!in->codes || !in->meta)) return fail(TC_ERR_NULL, "payload codes/meta is NULL");
    if (((uintptr_t)in->codes & 3u) != 0) return fail(TC_ERR_ALIGN, "codes must be 4-byte aligned");
    wire = -(int)c->bits;
  }
  TC_PRECONDITION(check_disjoint(
      {{in->idx, 4 * c->n_seg * c->k, "payload idx"},
       {c->kind == TC_TOPK ? in->val : nullptr, bytes_of(c->n_seg * c->k, c->wire), "payload val"},
       {c->kind == TC_TOPK_QUANT ? in->codes : nullptr, c->n_seg * tc_quant_group_bytes(c->k, c->bits), "codes"},
       {c->kind == TC_TOPK_QUANT ? in->meta : nullptr, 8 * c->n_seg, "meta"},
       {in->blk, 4 * c->n_seg * (tc::n_blocks(c->seg_len) + 1), "payload blk"},
       {y, bytes_of(c->n_seg * c->seg_len, out_dt), "output"}}));
  tc::ScatterArgs a{};
  a.idx = in->idx;
  a.blk = in->blk;
  a.val = in->val;
  a.codes = (const uint32_t*)in->codes;
  a.meta = in->meta;
  a.y = y;
  a.n_seg = c->n_seg;
  a.L = c->seg_len;
  a.k = c->k;
  a.wpg = (c->kind == TC_TOPK_QUANT) ? tc_quant_group_bytes(c->k, c->bits) / 4u : 0u;
  hipError_t he = tc::launch_topk_decompress(wire, out_dt, a, (hipStream_t)stream);
  if (he != hipSuccess) return hip_fail(he, "topk decompress launch");
  return TC_OK;
}

TC_API tc_status tc_topk_gather(const tc_codec* c, const tc_payload* in, const void* x, int dt, float* e,
                                void* val, void* stream) {
  tc_status s = check_codec(c, 1 << TC_TOPK);
  if (s != TC_OK) return s;
  if (!dt_ok(dt)) return fail(TC_ERR_DTYPE, "dtype %d", dt);
  if (c->wire != dt) return fail(TC_ERR_DTYPE, "wire dtype %d must equal the input dtype %d", c->wire, dt);
  if (c->n_seg * c->seg_len == 0) return TC_OK;
  if (!x) return fail(TC_ERR_NULL, "input is NULL");
  if (c->k > 0 && (!in || !in->idx || !val)) return fail(TC_ERR_NULL, "indices or val is NULL");
  TC_PRECONDITION(check_disjoint({{c->k > 0 ? in->idx : nullptr, 4 * c->n_seg * c->k, "payload idx"},
                                  {c->k > 0 ? in->blk : nullptr, 4 * c->n_seg * (tc::n_blocks(c->seg_len) + 1),
                                   "payload blk"},
                                  {x, bytes_of(c->n_seg * c->seg_len, dt), "input"},
                                  {e, 4 * c->n_seg * c->seg_len, "e"},
                                  {val, bytes_of(c->n_seg * c->k, dt), "val"}}));
  TC_PRECONDITION(check_values(dt, x, e, c->n_seg * c->seg_len, stream));
  if (c->k == 0 && !e) return TC_OK;
  tc::GatherArgs a{};
  a.idx = (c->k > 0) ? in->idx : nullptr;
  a.blk = (c->k > 0 && in) ? in->blk : nullptr;
  a.x = x;
  a.e = e;
  a.val = val;
  a.n_seg = c->n_seg;
  a.L = c->seg_len;
  a.k = c->k;
  hipError_t he = tc::launch_gather(dt, a, (hipStream_t)stream);
  if (he != hipSuccess) return hip_fail(he, "topk gather launch");
  return TC_OK;
}

TC_API tc_status tc_quant_pack(const tc_codec* c, const void* x, int dt, const tc_payload* out, void* ws,
                               size_t ws_bytes, void* stream) {
  tc_status s = check_codec(c, 1 << TC_QUANT);
  if (s != TC_OK) return s;
  return quant_common(false, c, x, dt, nullptr, out, ws, ws_bytes, stream);
}

TC_API tc_status tc_quant_unpack(const tc_codec* c, const tc_payload* in, void* y, int out_dt, void* stream) {
  tc_status s = check_codec(c, 1 << TC_QUANT);
  if (s != TC_OK) return s;
  if (!dt_ok(out_dt)) return fail(TC_ERR_DTYPE, "out dtype %d", out_dt);
  if (!in) return fail(TC_ERR_NULL, "payload is NULL");
  if (c->n_seg * c->seg_len == 0) return TC_OK;
  if (!y || !in->codes || !in->meta) return fail(TC_ERR_NULL, "output, codes or meta is NULL");
  if (((uintptr_t)in->codes & 3u) != 0) return fail(TC_ERR_ALIGN, "codes must be 4-byte aligned");
  TC_PRECONDITION(check_disjoint({{in->codes, c->n_seg * tc_quant_group_bytes(c->seg_len, c->bits), "codes"},
                                  {in->meta, 8 * c->n_seg, "meta"},
                                  {y, bytes_of(c->n_seg * c->seg_len, out_dt), "output"}}));
  tc::UnpackArgs a{};
  a.codes = (const uint32_t*)in->codes;
  a.meta = in->meta;
  a.y = y;
  a.n_grp = c->n_seg;
  a.G = c->seg_len;
  a.wpg = tc_quant_group_bytes(c->seg_len, c->bits) / 4u;
  hipError_t he = tc::launch_unpack(out_dt, c->bits, a, (hipStream_t)stream);
  if (he != hipSuccess) return hip_fail(he, "quant unpack launch");
  return TC_OK;
}

TC_API tc_status tc_ef_step(const tc_codec* c, const void* x, int dt, float* e, const tc_payload* out, void* ws,
                            size_t ws_bytes, void* stream) {
  tc_status s = check_codec(c, (1 << TC_TOPK) | (1 << TC_QUANT) | (1 << TC_TOPK_QUANT));
  if (s != TC_OK) return s;
  if (c->kind == TC_TOPK) return topk_common(tc::SEL_EF, c, x, dt, e, nullptr, 0, nullptr, out, ws, ws_bytes, stream);
  if (c->kind == TC_QUANT) return quant_common(true, c, x, dt, e, out, ws, ws_bytes, stream);
  // TopK, then the kept list quantized as one min-max group per segment
  if (!dt_ok(dt)) return fail(TC_ERR_DTYPE, "dtype %d", dt);
  if (c->wire != dt) return fail(TC_ERR_DTYPE, "wire (receiver) dtype %d must equal the input dtype %d", c->wire, dt);
  if (!out) return fail(TC_ERR_NULL, "payload is NULL");
  if (c->n_seg * c->seg_len == 0) return TC_OK;
  if (!x || !e) return fail(TC_ERR_NULL, "input or error buffer is NULL");
  if (c->k > 0 && (!out->idx || !out->codes || !out->meta)) return fail(TC_ERR_NULL, "payload idx/codes/meta is NULL");
  if (!out->meta) return fail(TC_ERR_NULL, "payload meta is NULL");
  if (((uintptr_t)out->codes & 3u) != 0) return fail(TC_ERR_ALIGN, "codes must be 4-byte aligned");
  const uint64_t n = c->n_seg * c->seg_len;
  TC_PRECONDITION(check_disjoint({{x, bytes_of(n, dt), "input"},
                                  {e, 4 * n, "e"},
                                  {out->idx, 4 * c->n_seg * c->k, "payload idx"},
                                  {out->codes, c->n_seg * tc_quant_group_bytes(c->k, c->bits), "codes"},
                                  {out->meta, 8 * c->n_seg, "meta"},
                                  {out->blk, 4 * c->n_seg * (tc::n_blocks(c->seg_len) + 1), "payload blk"},
                                  {ws, ws_bytes, "workspace"}}));
  TC_PRECONDITION(check_values(dt, x, e, n, stream));
  return global_topk(c->bits, c, x, dt, e, out, ws, ws_bytes, stream);
}

TC_API tc_status tc_efmix_step(const tc_codec* c, const void* x, int dt, float* e, const tc_payload* out_x,
                               const tc_payload* out_e, void* stream) {
  tc_status s = check_codec(c, 1 << TC_TOPK);
  if (s != TC_OK) return s;
  if (!dt_ok(dt)) return fail(TC_ERR_DTYPE, "dtype %d", dt);
  if (c->wire != dt) return fail(TC_ERR_DTYPE, "wire dtype %d must equal the input dtype %d", c->wire, dt);
  if (!out_x || !out_e) return fail(TC_ERR_NULL, "payload is NULL");
  if (c->n_seg * c->seg_len == 0) return TC_OK;
  if (c->seg_len > tc::LDS_SEG_MAX)
    return fail(TC_ERR_ARG, "EF-mixed segments hold at most %llu elements (got %llu)",
                (unsigned long long)tc::LDS_SEG_MAX, (unsigned long long)c->seg_len);
  if (!x || !e) return fail(TC_ERR_NULL, "input or error buffer is NULL");
  uint64_t kx = 0, ke = 0;
  tc_efmix_counts(c->k, &kx, &ke);
  if (kx > 0 && (!out_x->idx || !out_x->val)) return fail(TC_ERR_NULL, "input list idx/val is NULL");
  if (ke > 0 && (!out_e->idx || !out_e->val)) return fail(TC_ERR_NULL, "buffer list idx/val is NULL");
  const uint64_t n = c->n_seg * c->seg_len, nb = tc::n_blocks(c->seg_len) + 1;
  TC_PRECONDITION(check_disjoint({{x, bytes_of(n, dt), "input"},
                                  {e, 4 * n, "e"},
                                  {out_x->idx, 4 * c->n_seg * kx, "input list idx"},
                                  {out_x->val, bytes_of(c->n_seg * kx, dt), "input list val"},
                                  {out_x->blk, 4 * c->n_seg * nb, "input list blk"},
                                  {out_e->idx, 4 * c->n_seg * ke, "buffer list idx"},
                                  {out_e->val, bytes_of(c->n_seg * ke, dt), "buffer list val"},
                                  {out_e->blk, 4 * c->n_seg * nb, "buffer list blk"}}));
  TC_PRECONDITION(check_values(dt, x, e, n, stream));
  // the two selections (two workgroups per segment), then the residual
  const tc::SegPlan p = tc::plan_lds(tc::SEL_EFMIX, dt, 2 * c->n_seg);
  tc::TopkArgs a{};
  a.x = x;
  a.e = e;
  a.idx = out_x->idx;
  a.val = out_x->val;
  a.blk = out_x->blk;
  a.k = kx;
  a.idx2 = out_e->idx;
  a.val2 = out_e->val;
  a.blk2 = out_e->blk;
  a.k2 = ke;
  a.n_seg = c->n_seg;
  a.L = c->seg_len;
  hipError_t he = tc::launch_topk(tc::SEL_EFMIX, dt, p, a, (hipStream_t)stream);
  if (he != hipSuccess) return hip_fail(he, "efmix launch");
  tc::EfmixResidArgs r{};
  r.x = x;
  r.e = e;
  r.idx = out_x->idx;
  r.blk = out_x->blk;
  r.idx2 = out_e->idx;
  r.blk2 = out_e->blk;
  r.n_seg = c->n_seg;
  r.L = c->seg_len;
  r.k = kx;
  r.k2 = ke;
  he = tc::launch_efmix_resid(dt, r, (hipStream_t)stream);
  if (he != hipSuccess) return hip_fail(he, "efmix residual launch");
  return TC_OK;
}

TC_API tc_status tc_efmix_reconstruct(const tc_codec* c, const tc_payload* in_x, const tc_payload* in_e, void* y,
                                      int out_dt, void* stream) {
  tc_status s = check_codec(c, 1 << TC_TOPK);
  if (s != TC_OK) return s;
  if (!dt_ok(c->wire)) return fail(TC_ERR_DTYPE, "wire dtype %d", c->wire);
  if (!dt_ok(out_dt)) return fail(TC_ERR_DTYPE, "out dtype %d", out_dt);
  if (!in_x || !in_e) return fail(TC_ERR_NULL, "payload is NULL");
  if (c->n_seg * c->seg_len == 0) return TC_OK;
  if (!y) return fail(TC_ERR_NULL, "output is NULL");
  uint64_t kx = 0, ke = 0;
  tc_efmix_counts(c->k, &kx, &ke);
  if (kx > 0 && (!in_x->idx || !in_x->val)) return fail(TC_ERR_NULL, "input list idx/val is NULL");
  if (ke > 0 && (!in_e->idx || !in_e->val)) return fail(TC_ERR_NULL, "buffer list idx/val is NULL");
  const uint64_t nb = tc::n_blocks(c->seg_len) + 1;
  TC_PRECONDITION(check_disjoint({{in_x->idx, 4 * c->n_seg * kx, "input list idx"},
                                  {in_x->val, bytes_of(c->n_seg * kx, c->wire), "input list val"},
                                  {in_x->blk, 4 * c->n_seg * nb, "input list blk"},
                                  {in_e->idx, 4 * c->n_seg * ke, "buffer list idx"},
                                  {in_e->val, bytes_of(c->n_seg * ke, c->wire), "buffer list val"},
                                  {in_e->blk, 4 * c->n_seg * nb, "buffer list blk"},
                                  {y, bytes_of(c->n_seg * c->seg_len, out_dt), "output"}}));
  tc::ScatterArgs a{};
  a.idx = in_x->idx;
  a.blk = in_x->blk;
  a.val = in_x->val;
  a.k = kx;
  a.idx2 = in_e->idx;
  a.blk2 = in_e->blk;
  a.val2 = in_e->val;
  a.k2 = ke;
  a.y = y;
  a.n_seg = c->n_seg;
  a.L = c->seg_len;
  hipError_t he = tc::launch_efmix_recv(c->wire, out_dt, a, (hipStream_t)stream);
  if (he != hipSuccess) return hip_fail(he, "efmix reconstruct launch");
  return TC_OK;
}

TC_API tc_status tc_aqsgd_step(const tc_codec* c, const void* a, int dt, void* m, uint64_t n_samples,
                               const int64_t* ids, uint32_t n_ids, const tc_payload* out, void* ws,
                               size_t ws_bytes, void* stream) {
  const tc_status s = check_aqsgd_args(c, n_samples, n_ids);
  if (s != TC_OK) return s;
  return topk_common(tc::SEL_AQSGD, c, a, dt, nullptr, m, n_samples, ids, out, ws, ws_bytes, stream);
}

TC_API tc_status tc_aqsgd_step_noalloc(const tc_codec* c, const void* a, int dt, void* m, uint64_t n_samples,
                                       const int64_t* ids, uint32_t n_ids, const tc_payload* out, void* stream) {
  const tc_status s = check_aqsgd_args(c, n_samples, n_ids);
  if (s != TC_OK) return s;
  return topk_common(tc::SEL_AQSGD, c, a, dt, nullptr, m, n_samples, ids, out, nullptr, 0, stream, true);
}

TC_API tc_status tc_aqsgd_reconstruct(const tc_codec* c, const tc_payload* in, void* m_r, int dt, uint64_t n_samples,
                                      const int64_t* ids, uint32_t n_ids, void* a_hat, void* stream) {
  tc_status s = check_codec(c, 1 << TC_TOPK);
  if (s != TC_OK) return s;
  if (!dt_ok(dt)) return fail(TC_ERR_DTYPE, "dtype %d", dt);
  if (c->wire != dt) return fail(TC_ERR_DTYPE, "wire dtype %d must equal the buffer dtype %d", c->wire, dt);
  if (c->n_seg != n_ids) return fail(TC_ERR_ARG, "codec.n_seg %llu != n_ids %u", (unsigned long long)c->n_seg, n_ids);
  if (!in) return fail(TC_ERR_NULL, "payload is NULL");
  if (c->n_seg * c->seg_len == 0) return TC_OK;
  if (n_samples == 0) return fail(TC_ERR_ARG, "n_samples is 0");
  if (c->seg_len != 0 && n_samples > UINT64_MAX / c->seg_len) return fail(TC_ERR_ARG, "n_samples * seg_len overflows");
  if (!m_r || !ids || !a_hat) return fail(TC_ERR_NULL, "buffer, ids or output is NULL");
  if (c->k > 0 && (!in->idx || !in->val)) return fail(TC_ERR_NULL, "payload idx/val is NULL");
  TC_PRECONDITION(check_disjoint({{in->idx, 4 * c->n_seg * c->k, "payload idx"},
                                  {in->val, bytes_of(c->n_seg * c->k, dt), "payload val"},
                                  {in->blk, 4 * c->n_seg * (tc::n_blocks(c->seg_len) + 1), "payload blk"},
                                  {m_r, bytes_of(n_samples * c->seg_len, dt), "m_r"},
                                  {ids, 8 * c->n_seg, "ids"},
                                  {a_hat, bytes_of(c->n_seg * c->seg_len, dt), "output"}}));
  TC_PRECONDITION(check_ids_distinct(ids, c->n_seg, stream));
  tc::ScatterArgs a{};
  a.idx = in->idx;
  a.blk = in->blk;
  a.val = in->val;
  a.y = a_hat;
  a.m = m_r;
  a.ids = ids;
  a.n_samples = n_samples;
  a.n_seg = c->n_seg;
  a.L = c->seg_len;
  a.k = c->k;
  hipError_t he = tc::launch_aqsgd_recv(dt, a, (hipStream_t)stream);
  if (he != hipSuccess) return hip_fail(he, "aqsgd reconstruct launch");
  return TC_OK;
}
