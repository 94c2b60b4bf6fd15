/*
 * tc.h -- C ABI of libtc, the MI355X (gfx950) boundary compressors for
 * model-parallel training, after
 *   M. Rudakov, A. Beznosikov, Y. Kholodov, A. Gasnikov,
 *   "Activations and Gradients Compression for Model-Parallel Training".
 *
 * Every tensor that crosses a pipeline-stage boundary (activations forward,
 * their gradients backward; paper Sec. 2.1, Fig. 1) is compressed by the
 * sender and decompressed by the receiver.  This library implements both
 * sides for:
 *   - TopK sparsification (Sec. 2.3) as an index + value payload;
 *   - uniform b-bit min-max quantization with bit packing (Sec. 2.2);
 *   - error feedback around either compressor (Sec. 2.4);
 *   - AQ-SGD per-example error feedback with TopK (Sec. 2.5).
 *
 * Conventions shared by every entry point
 *   Memory    All tensor pointers are device pointers (hipMalloc or a torch
 *             tensor's data).  The caller allocates and owns every buffer;
 *             the library allocates no device memory and keeps no pointer
 *             after a call returns.  The one exception is the scratch array
 *             of tc_aqsgd_step_noalloc, a fixed-size device global of the
 *             library itself.
 *   Streams   `stream` is a hipStream_t (NULL = the default stream).  Work is
 *             enqueued asynchronously; TC_OK means "enqueued".  Kernel-side
 *             faults in the data (an out-of-range sample id or payload index,
 *             a cross-workgroup wait that timed out) are recorded in sticky
 *             per-device bits read by tc_device_errors().
 *   Errors    Arguments are validated on the host before anything is
 *             enqueued; on error nothing is enqueued and no output is touched.
 *             tc_last_error() returns a thread-local description.
 *   Layout    Row-major.  A "segment" is one independent unit of compression
 *             (a sample [C*H*W], a token row [H], or a whole tensor [N]):
 *             x is [n_seg][seg_len].  Payload arrays are [n_seg][k].
 *   Dtypes    Inputs are TC_F32, TC_BF16 or TC_F16.  Widening to binary32 is
 *             exact; every narrowing rounds to nearest, ties to even.  All
 *             arithmetic is IEEE binary32 without contraction into FMA.
 *   Workspace Kernels that spread one segment over several workgroups keep
 *             small counters in a caller-owned, 8-byte aligned workspace of
 *             tc_workspace_bytes() bytes.  It must be zero-filled before its
 *             first use; every completed call leaves it zero-filled again.
 *             After tc_device_errors() reports TC_KERR_TIMEOUT it must be
 *             zero-filled again.  Calls that run concurrently need distinct
 *             workspaces.  The size depends on the codec and on the current
 *             device.
 *   Co-residency  Such kernels wait for each other inside one launch.  They
 *             are sized to fit the device at once, and their waits are
 *             bounded (TC_KERR_TIMEOUT), but two of them should not share the
 *             device with other long-running kernels on concurrent streams.
 *             Once TC_KERR_TIMEOUT is set on a device, every later such
 *             kernel gives up its waits early and its results are invalid
 *             until tc_device_errors(..., clear = 1) resets the bit and the
 *             workspaces are zero-filled again.
 *   Preconditions  The release library (libtc.so) assumes, without checking:
 *             finite inputs, |x + e| at most half the binary32 maximum (so
 *             that a quantization range hi - lo is finite), AQ-SGD changes
 *             a - m[id] and updated values m[id] + v that fit the buffer's
 *             dtype, distinct AQ-SGD ids within one call (two workgroups
 *             would otherwise update one buffer row at once), and no overlap
 *             between any two of a call's buffers (e and m are in-out on
 *             their own).  The debug library (libtc_debug.so, the same
 *             sources built with TC_DEBUG) checks all of these before the
 *             launch and returns TC_ERR_PRECONDITION, with nothing enqueued,
 *             when one fails.  Its checks read device data and synchronize
 *             the stream, so its calls cannot be captured into a graph.
 */
#ifndef TC_H
#define TC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TC_OK = 0,
  TC_ERR_NULL = 1,       /* a required pointer is NULL */
  TC_ERR_ARG = 2,        /* a size, count or kind is out of range */
  TC_ERR_DTYPE = 3,      /* dtype not supported for this operation */
  TC_ERR_WORKSPACE = 4,  /* workspace missing or smaller than tc_workspace_bytes() */
  TC_ERR_HIP = 5,        /* the HIP runtime refused the launch (see tc_last_error) */
  TC_ERR_PRECONDITION = 6, /* debug library only: an assumption below does not hold */
  TC_ERR_ALIGN = 7       /* a code buffer or the workspace is misaligned */
} tc_status;

typedef enum { TC_F32 = 0, TC_BF16 = 1, TC_F16 = 2 } tc_dtype;

typedef enum {
  TC_TOPK = 1,        /* TopK: idx + val payload */
  TC_QUANT = 2,       /* min-max quantization: codes + meta payload */
  TC_TOPK_QUANT = 3   /* TopK, then the kept list quantized as one group per segment */
} tc_kind;

/* kernel-side error bits reported by tc_device_errors() */
#define TC_KERR_TIMEOUT 1u    /* a cross-workgroup wait gave up; results and workspace invalid */
#define TC_KERR_BAD_ID 2u     /* an AQ-SGD sample id was outside [0, n_samples); that row was skipped */
#define TC_KERR_BAD_INDEX 4u  /* a payload index lay outside its segment; the entry was skipped */
#define TC_KERR_INTERNAL 8u   /* a selection placed more than k entries (a library fault); extra entries dropped */

/* What one compression operator does to a tensor of n_seg * seg_len elements.
 *   kind     tc_kind
 *   wire     dtype of TopK values on the wire; must equal the input dtype
 *   bits     TC_QUANT / TC_TOPK_QUANT: 1..8 bits per code, or 32 = values
 *            sent as binary32 (no compression)
 *   n_seg    segments (TopK) or quantization groups (TC_QUANT)
 *   seg_len  elements per segment / group, < 2^32
 *   k        TopK: entries kept per segment, 0 <= k <= seg_len
 *            (tc_topk_count() turns "K percent" into k)                    */
typedef struct {
  int32_t kind;
  int32_t wire;
  uint32_t bits;
  uint32_t reserved;   /* must be 0 */
  uint64_t n_seg;
  uint64_t seg_len;
  uint64_t k;
} tc_codec;

/* Length of the index blocks of a TopK payload's block table (see blk). */
#define TC_BLOCK_LEN 4096u

/* The message a sender produces.  Unused members may be NULL.
 *   idx    TC_TOPK, TC_TOPK_QUANT: [n_seg][k] uint32 indices within the
 *          segment, strictly ascending
 *   val    TC_TOPK: [n_seg][k] kept values in the wire dtype
 *   codes  TC_QUANT: [n_seg][tc_quant_group_bytes(seg_len, bits)] bytes;
 *          TC_TOPK_QUANT: [n_seg][tc_quant_group_bytes(k, bits)]; codes are
 *          packed LSB-first into little-endian 32-bit words (4-byte aligned)
 *   meta   TC_QUANT, TC_TOPK_QUANT: [n_seg][2] binary32 (lo, scale); the
 *          receiver reconstructs lo + code * scale
 *   blk    TC_TOPK, TC_TOPK_QUANT, optional: [n_seg][ceil(seg_len /
 *          TC_BLOCK_LEN) + 1] uint32; blk[s][b] = number of kept entries of
 *          segment s with index < b * TC_BLOCK_LEN (so blk[s][0] = 0 and the
 *          last entry is k).  A sender writes it when non-NULL; a receiver
 *          given it reads each block's entries directly instead of searching
 *          idx.  4 bytes per 4096 elements.                                  */
typedef struct {
  uint32_t* idx;
  void* val;
  uint8_t* codes;
  float* meta;
  uint32_t* blk;
} tc_payload;

/* ---------------------------------------------------------------- helpers */

/* Sec. 2.3 "K%": entries kept out of seg_len for the fraction num/den, the
 * exact ceiling of seg_len*num/den in integer arithmetic (0 if den == 0). */
uint64_t tc_topk_count(uint64_t seg_len, uint32_t num, uint32_t den);

/* Sec. 2.2: bytes of one group's packed codes: 4*ceil(grp_len*bits/32) for
 * bits in 1..8, 4*grp_len for bits == 32, 0 otherwise. */
uint64_t tc_quant_group_bytes(uint64_t grp_len, uint32_t bits);

/* Workspace bytes any call with this codec needs on the current device (may
 * be 0, in which case ws may be NULL). */
tc_status tc_workspace_bytes(const tc_codec* c, size_t* bytes);

/* Static description of a status code. */
const char* tc_status_str(int status);

/* Thread-local description of the last error returned on this thread. */
const char* tc_last_error(void);

/* Synchronizes the current device, then reports (and if `clear`, resets) the
 * sticky TC_KERR_* bits of the kernels run on it. */
tc_status tc_device_errors(uint32_t* bits, int clear);

/* For tests of the recovery path: synchronizes the current device and ORs
 * `bits` (TC_KERR_* only, else TC_ERR_ARG) into its sticky bits, as a kernel
 * would.  With TC_KERR_TIMEOUT set, every later cross-workgroup wait gives up
 * after about a thousand polls instead of its full bound (a wait its group
 * satisfies sooner completes as usual); results are invalid until the bit is
 * cleared and the workspaces are zero-filled again, as after a real timeout. */
tc_status tc_raise_device_errors(uint32_t bits);

/* ------------------------------------------------------------------ TopK */

/* Sec. 2.3 sender: per segment, the k entries of x with the largest |x|; ties
 * in |x| (including +0 against -0) go to the lower index.  Writes out->idx
 * (ascending) and out->val (x itself at those indices, in the wire dtype).
 * x: [n_seg][seg_len] of dtype dt.  kind must be TC_TOPK. */
tc_status tc_topk_compress(const tc_codec* c, const void* x, int dt, const tc_payload* out,
                           void* ws, size_t ws_bytes, void* stream);

/* Sec. 2.3 receiver: y [n_seg][seg_len] of dtype out_dt, +0 everywhere except
 * y[s][idx[s][j]] = the sent value.  TC_TOPK reads in->idx/val; TC_TOPK_QUANT
 * reads in->idx/codes/meta and writes lo + code_j*scale at idx_j.  in->blk,
 * when non-NULL, is the sender's block table (it gives each chunk its range;
 * for segments of up to 2048 elements it is only checked).  An index outside
 * its segment, a list that is not strictly ascending where the range comes
 * from a search (or, for segments of up to 2048 elements, anywhere), or a
 * block table that does not fit the list is reported by tc_device_errors;
 * the rest of the tensor is still written. */
tc_status tc_topk_decompress(const tc_codec* c, const tc_payload* in, void* y, int out_dt, void* stream);

/* Sec. 3.2 (the GPT-2 runs, Table 5 and its note): gradients compressed at
 * the indices that the activations' TopK kept, instead of a selection of
 * their own (compressing them separately made those runs diverge).
 *   in->idx  [n_seg][k] strictly ascending indices within each segment, the
 *            idx of that TopK payload; in->blk, when non-NULL, its block
 *            table (used only with e)
 *   x        [n_seg][seg_len] of dtype dt (the gradient)
 *   val      [n_seg][k] output: x at those indices, in dt (the wire dtype)
 *   e        NULL, or the Sec. 2.4 residual [n_seg][seg_len] binary32, in-out:
 *            X = x + e is what is sent, and e <- X - r with r what the
 *            receiver's dense tensor holds (X's wire value at the indices, +0
 *            elsewhere)
 * The receiver is tc_topk_decompress with in->idx (and in->blk) and val.
 * kind must be TC_TOPK and wire == dt.  An index outside its segment sets
 * TC_KERR_BAD_INDEX and its entry is sent as +0 (with e, left unchanged in
 * the residual); with e and no block table, indices that do not ascend set
 * it too. */
tc_status tc_topk_gather(const tc_codec* c, const tc_payload* in, const void* x, int dt, float* e, void* val,
                         void* stream);

/* -------------------------------------------------------- quantization */

/* Sec. 2.2 sender: per group of seg_len elements, lo = min and hi = max (a
 * -0 reads as +0), code_i = min(rint((x_i - lo)/(hi - lo) * (2^bits - 1)),
 * 2^bits - 1) with round-half-even, scale = (hi - lo)/(2^bits - 1); a
 * constant group gets codes 0 and scale 0.  kind must be TC_QUANT.  Writes
 * out->codes and out->meta.  The receiver's dtype equals dt. */
tc_status tc_quant_pack(const tc_codec* c, const void* x, int dt, const tc_payload* out,
                        void* ws, size_t ws_bytes, void* stream);

/* Sec. 2.2 receiver: y [n_seg][seg_len] in out_dt, y_i = lo + code_i*scale
 * (product and sum each rounded to binary32), or the sent binary32 values
 * when bits == 32. */
tc_status tc_quant_unpack(const tc_codec* c, const tc_payload* in, void* y, int out_dt, void* stream);

/* ------------------------------------------------------- error feedback */

/* Sec. 2.4 sender with error feedback: X = x + e (binary32), send C(X), then
 * e <- X - r where r is exactly what the receiver's dense tensor will hold
 * (read back as binary32).  C is the codec's compressor (TopK, quantization,
 * or TopK whose kept list is quantized as one min-max group per segment,
 * TC_TOPK_QUANT).  e: [n_seg][seg_len] binary32, in-out, one buffer per
 * compression operator, zero at the first step.  Segments longer than one
 * resident group of workgroups holds (TC_TOPK) and every TC_TOPK_QUANT
 * segment run through a chain of kernels over the whole segment; they need
 * seg_len < 2^31. */
tc_status tc_ef_step(const tc_codec* c, const void* x, int dt, float* e, const tc_payload* out,
                     void* ws, size_t ws_bytes, void* stream);

/* Sec. 2.4, EF-mixed: half of the TopK budget k goes to the input, half to
 * the error buffer.  Per segment (binary32 arithmetic):
 *   (idx_x, v_x) = TopK(x, k_x),  k_x = k - floor(k/2), v_x sent in dt
 *   (idx_e, v_e) = TopK(e, k_e),  k_e = floor(k/2),     v_e = e rounded to dt
 *   e_i <- (x_i - [i in idx_x] v_x) + (e_i - [i in idx_e] v_e)
 * so e becomes x + e minus the sent tensor C(x) + C(e).  Both selections use
 * TopK's order (larger |v| first, ties to the lower index) and each list is in
 * ascending index order; the two lists may share indices.  x: [n_seg][seg_len]
 * dt; e: [n_seg][seg_len] binary32, in-out, zero at the first step; out_x holds
 * idx [n_seg][k_x], val [n_seg][k_x] (dt) and an optional block table; out_e
 * the same with k_e.  kind must be TC_TOPK with wire == dt; seg_len is at most
 * 32,768 (one workgroup holds the segment), else TC_ERR_ARG. */
tc_status tc_efmix_step(const tc_codec* c, const void* x, int dt, float* e, const tc_payload* out_x,
                        const tc_payload* out_e, void* stream);

/* Sec. 2.4, EF-mixed: how a budget of k entries splits between the input's
 * list (k_x = k - floor(k/2), the odd entry goes to the input) and the error
 * buffer's list (k_e = floor(k/2)).  Either output pointer may be NULL. */
void tc_efmix_counts(uint64_t k, uint64_t* k_x, uint64_t* k_e);

/* Sec. 2.4, EF-mixed receiver: y [n_seg][seg_len] in out_dt starts at +0,
 * takes v_x at idx_x, then adds v_e at idx_e (binary32 sum), rounded once to
 * out_dt.  Payload lists as tc_efmix_step writes them (wire dtype c->wire);
 * any seg_len.  An index outside its segment, or (without a block table) a
 * list that is not strictly ascending, is reported by tc_device_errors. */
tc_status tc_efmix_reconstruct(const tc_codec* c, const tc_payload* in_x, const tc_payload* in_e, void* y,
                               int out_dt, void* stream);

/* ---------------------------------------------------------------- AQ-SGD */

/* Sec. 2.5 sender with TopK: for each b < n_ids, with id = ids[b]:
 *   d = a[b] - m[id]                  (binary32)
 *   (idx, v) = TopK(d, k), v sent in dt
 *   m[id][idx_j] <- m[id][idx_j] + v_j  (rounded to dt)
 * a: [n_ids][seg_len] dt; m: [n_samples][seg_len] dt, in-out; ids: device
 * int64 [n_ids], distinct, in [0, n_samples).  kind must be TC_TOPK with
 * n_seg == n_ids. */
tc_status tc_aqsgd_step(const tc_codec* c, const void* a, int dt, void* m, uint64_t n_samples,
                        const int64_t* ids, uint32_t n_ids, const tc_payload* out, void* ws,
                        size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under stream or graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * tc_aqsgd_step above, with the same arguments and results bit for bit, but
 * without a workspace argument.  The kernels use instead a scratch array of
 * TC_NOALLOC_SCRATCH_BYTES that the library holds on each device it runs on
 * until the process ends; this call allocates nothing.  A shape that needs
 * more scratch than that fails with TC_ERR_WORKSPACE and nothing enqueued
 * (the need never exceeds tc_workspace_bytes()).  The first call on a device
 * looks up that device's copy and enqueues a clearing kernel on `stream`.
 * Every call on one device shares its scratch, so two calls that overlap in
 * time on one device (concurrent streams, host threads) race and both give
 * invalid results.  After TC_KERR_TIMEOUT, tc_device_errors(..., clear = 1)
 * clears the current device's scratch again. */
#define TC_NOALLOC_SCRATCH_BYTES (4u << 20)
tc_status tc_aqsgd_step_noalloc(const tc_codec* c, const void* a, int dt, void* m, uint64_t n_samples,
                                const int64_t* ids, uint32_t n_ids, const tc_payload* out, void* stream);

/* Sec. 2.5 receiver: applies the same update to its own copy m_r of the
 * buffer and writes the updated rows: a_hat[b] = m_r[ids[b]] after the
 * update.  m_r: [n_samples][seg_len] dt, in-out; a_hat: [n_ids][seg_len] dt.
 * An id outside [0, n_samples) skips its row and an index outside its
 * segment skips its entry; both are reported by tc_device_errors. */
tc_status tc_aqsgd_reconstruct(const tc_codec* c, const tc_payload* in, void* m_r, int dt,
                               uint64_t n_samples, const int64_t* ids, uint32_t n_ids, void* a_hat,
                               void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TC_H */
