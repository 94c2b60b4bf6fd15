"""Python binding of libtc (include/tc.h): argument marshalling only.

Each function takes torch tensors that already live on the GPU, allocates the
outputs with torch (device memory and the current stream are all torch is used
for), and calls the C entry point of the same name.  Every step of the
compression runs in the HIP kernels of libtc.so; there is no fallback: if the
library is missing or no GPU is present, the calls raise.
"""
from __future__ import annotations

import ctypes as C
import os
import threading
from typing import NamedTuple, Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtc.so")
# the same library with its preconditions checked before every launch
# (TC_ERR_PRECONDITION); chosen with use_debug_library() or TC_DEBUG=1
DEBUG_LIB_PATH = os.path.join(_HERE, "libtc_debug.so")
(TC_OK, TC_ERR_NULL, TC_ERR_ARG, TC_ERR_DTYPE, TC_ERR_WORKSPACE, TC_ERR_HIP, TC_ERR_PRECONDITION,
 TC_ERR_ALIGN) = range(8)

TC_F32, TC_BF16, TC_F16 = 0, 1, 2
TC_TOPK, TC_QUANT, TC_TOPK_QUANT = 1, 2, 3
TC_KERR_TIMEOUT, TC_KERR_BAD_ID, TC_KERR_BAD_INDEX, TC_KERR_INTERNAL = 1, 2, 4, 8

_DT = {torch.float32: TC_F32, torch.bfloat16: TC_BF16, torch.float16: TC_F16}
_TORCH = {v: k for k, v in _DT.items()}


class Codec(C.Structure):
    _fields_ = [("kind", C.c_int32), ("wire", C.c_int32), ("bits", C.c_uint32), ("reserved", C.c_uint32),
                ("n_seg", C.c_uint64), ("seg_len", C.c_uint64), ("k", C.c_uint64)]


class Payload(C.Structure):
    _fields_ = [("idx", C.c_void_p), ("val", C.c_void_p), ("codes", C.c_void_p), ("meta", C.c_void_p),
                ("blk", C.c_void_p)]


BLOCK_LEN = 4096   # TC_BLOCK_LEN


def n_blocks(seg_len: int) -> int:
    return (seg_len + BLOCK_LEN - 1) // BLOCK_LEN


class TopkPayload(NamedTuple):
    """a TopK message: indices (uint32 patterns in an int32 tensor), values,
    and the block table ([n_seg, n_blocks + 1] int32, or None)"""
    idx: torch.Tensor
    val: torch.Tensor
    blk: Optional[torch.Tensor]


def empty_topk_payload(n_seg: int, seg_len: int, k: int, dtype, device, blk: bool = True) -> TopkPayload:
    return TopkPayload(torch.empty((n_seg, k), dtype=torch.int32, device=device),
                       torch.empty((n_seg, k), dtype=dtype, device=device),
                       torch.empty((n_seg, n_blocks(seg_len) + 1), dtype=torch.int32, device=device) if blk else None)


class TCError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: {status_str(status)} ({detail})")
        self.status = status


_lib = None
_lock = threading.Lock()

EXPORTS = {
    # name: (restype, argtypes)
    "tc_topk_count": (C.c_uint64, [C.c_uint64, C.c_uint32, C.c_uint32]),
    "tc_quant_group_bytes": (C.c_uint64, [C.c_uint64, C.c_uint32]),
    "tc_workspace_bytes": (C.c_int, [C.POINTER(Codec), C.POINTER(C.c_size_t)]),
    "tc_status_str": (C.c_char_p, [C.c_int]),
    "tc_last_error": (C.c_char_p, []),
    "tc_device_errors": (C.c_int, [C.POINTER(C.c_uint32), C.c_int]),
    "tc_topk_compress": (C.c_int, [C.POINTER(Codec), C.c_void_p, C.c_int, C.POINTER(Payload), C.c_void_p,
                                   C.c_size_t, C.c_void_p]),
    "tc_topk_decompress": (C.c_int, [C.POINTER(Codec), C.POINTER(Payload), C.c_void_p, C.c_int, C.c_void_p]),
    "tc_topk_gather": (C.c_int, [C.POINTER(Codec), C.POINTER(Payload), C.c_void_p, C.c_int, C.POINTER(C.c_float),
                                 C.c_void_p, C.c_void_p]),
    "tc_quant_pack": (C.c_int, [C.POINTER(Codec), C.c_void_p, C.c_int, C.POINTER(Payload), C.c_void_p,
                                C.c_size_t, C.c_void_p]),
    "tc_quant_unpack": (C.c_int, [C.POINTER(Codec), C.POINTER(Payload), C.c_void_p, C.c_int, C.c_void_p]),
    "tc_ef_step": (C.c_int, [C.POINTER(Codec), C.c_void_p, C.c_int, C.POINTER(C.c_float), C.POINTER(Payload),
                             C.c_void_p, C.c_size_t, C.c_void_p]),
    "tc_efmix_step": (C.c_int, [C.POINTER(Codec), C.c_void_p, C.c_int, C.POINTER(C.c_float), C.POINTER(Payload),
                                C.POINTER(Payload), C.c_void_p]),
    "tc_efmix_reconstruct": (C.c_int, [C.POINTER(Codec), C.POINTER(Payload), C.POINTER(Payload), C.c_void_p, C.c_int,
                                       C.c_void_p]),
    "tc_aqsgd_step": (C.c_int, [C.POINTER(Codec), C.c_void_p, C.c_int, C.c_void_p, C.c_uint64, C.c_void_p,
                                C.c_uint32, C.POINTER(Payload), C.c_void_p, C.c_size_t, C.c_void_p]),
    "tc_raise_device_errors": (C.c_int, [C.c_uint32]),
    "tc_aqsgd_step_noalloc": (C.c_int, [C.POINTER(Codec), C.c_void_p, C.c_int, C.c_void_p, C.c_uint64,
                                        C.c_void_p, C.c_uint32, C.POINTER(Payload), C.c_void_p]),
    "tc_aqsgd_reconstruct": (C.c_int, [C.POINTER(Codec), C.POINTER(Payload), C.c_void_p, C.c_int, C.c_uint64,
                                       C.c_void_p, C.c_uint32, C.c_void_p, C.c_void_p]),
    "tc_efmix_counts": (None, [C.c_uint64, C.POINTER(C.c_uint64), C.POINTER(C.c_uint64)]),
}


_loaded = {}
_debug = os.environ.get("TC_DEBUG", "") not in ("", "0")


def load(path: str):
    """load one build of the library with the prototypes of include/tc.h"""
    with _lock:
        L = _loaded.get(path)
        if L is None:
            if not os.path.exists(path):
                raise RuntimeError(f"{path} is missing: build it with paper_2401_07788_amd.build.build()")
            L = C.CDLL(path)
            for name, (res, args) in EXPORTS.items():
                f = getattr(L, name)
                f.restype = res
                f.argtypes = args
            _loaded[path] = L
    return L


def lib():
    """the library every call of this module goes through: libtc.so, or
    libtc_debug.so after use_debug_library(True) (raises if it is not built)"""
    global _lib
    if _lib is None:
        _lib = load(DEBUG_LIB_PATH if _debug else LIB_PATH)
    return _lib


def use_debug_library(on: bool = True) -> bool:
    """route later calls to the debug library (preconditions checked before
    each launch) or back to the release library; returns the previous choice"""
    global _lib, _debug
    prev = _debug
    _debug = bool(on)
    _lib = None
    return prev


def status_str(s: int) -> str:
    return lib().tc_status_str(s).decode()


def _check(rc: int, where: str):
    if rc != 0:
        raise TCError(rc, where, lib().tc_last_error().decode())


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(device):
    return C.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _need_gpu(*ts):
    for t in ts:
        if t is not None:
            if not t.is_cuda:
                raise ValueError("libtc works on GPU tensors only")
            if not t.is_contiguous():
                raise ValueError("libtc needs contiguous tensors")


def _check_topk_payload(pl, n_seg: int, k: int, seg_len: int, val_dtype, device, what: str = "payload",
                        need_val: bool = True):
    """a TopK payload the caller supplies must have exactly the shapes the
    kernels write or read: the C entry points only see pointers"""
    if pl.idx is None or tuple(pl.idx.shape) != (n_seg, k) or pl.idx.dtype != torch.int32:
        raise ValueError(f"{what}.idx must be int32 [{n_seg}, {k}]")
    if need_val:
        if pl.val is None or tuple(pl.val.shape) != (n_seg, k):
            raise ValueError(f"{what}.val must be [{n_seg}, {k}]")
        if pl.val.dtype != val_dtype:
            raise TypeError(f"{what}.val must be {val_dtype}")
    if pl.blk is not None and (tuple(pl.blk.shape) != (n_seg, n_blocks(seg_len) + 1) or pl.blk.dtype != torch.int32):
        raise ValueError(f"{what}.blk must be int32 [{n_seg}, {n_blocks(seg_len) + 1}]")
    for t in (pl.idx, pl.val if need_val else None, pl.blk):
        if t is not None and (t.device != device or not t.is_contiguous()):
            raise ValueError(f"{what} tensors must be contiguous on {device}")


def _segments(x: torch.Tensor, n_seg: int) -> int:
    """segment length of x viewed as [n_seg, seg_len]"""
    if n_seg <= 0 or x.numel() % n_seg != 0:
        raise ValueError(f"{x.numel()} elements do not split into {n_seg} segments")
    return x.numel() // n_seg


def _dt(t) -> int:
    try:
        return _DT[t.dtype]
    except KeyError:
        raise TypeError(f"unsupported dtype {t.dtype}") from None


def codec(kind: int, n_seg: int, seg_len: int, k: int = 0, bits: int = 0, wire: int = TC_F32) -> Codec:
    return Codec(kind, wire, bits, 0, n_seg, seg_len, k)


# ------------------------------------------------------------------ helpers
def topk_count(seg_len: int, num: int, den: int) -> int:
    return int(lib().tc_topk_count(seg_len, num, den))


def quant_group_bytes(grp_len: int, bits: int) -> int:
    return int(lib().tc_quant_group_bytes(grp_len, bits))


def workspace_bytes(c: Codec) -> int:
    n = C.c_size_t(0)
    _check(lib().tc_workspace_bytes(C.byref(c), C.byref(n)), "tc_workspace_bytes")
    return int(n.value)


_ws_cache = {}


def workspace(c: Codec, device=None) -> torch.Tensor | None:
    """a zero-filled workspace for this codec, reused across calls on one device
    and stream (every completed call leaves it zero-filled again)"""
    device = torch.device(device or torch.cuda.current_device())
    n = workspace_bytes(c)
    if n == 0:
        return None
    key = (device.index, torch.cuda.current_stream(device).cuda_stream)
    ws = _ws_cache.get(key)
    if ws is None or ws.numel() < n:
        ws = torch.zeros(max(n, 1 << 16), dtype=torch.uint8, device=device)
        _ws_cache[key] = ws
    return ws


def device_errors(clear: bool = True) -> int:
    """sticky TC_KERR_* bits of the current device (synchronizes it).  After a
    timed-out cross-workgroup wait the cached workspaces are zero-filled again."""
    bits = C.c_uint32(0)
    _check(lib().tc_device_errors(C.byref(bits), int(clear)), "tc_device_errors")
    if bits.value & TC_KERR_TIMEOUT:
        for ws in _ws_cache.values():
            ws.zero_()
        torch.cuda.synchronize()
    return int(bits.value)


def raise_device_errors(bits: int) -> None:
    """set sticky TC_KERR_* bits on the current device from the host, as a
    kernel would (tests of the recovery path)"""
    _check(lib().tc_raise_device_errors(int(bits)), "tc_raise_device_errors")


def _ws_args(c, device, ws):
    if ws is None:
        ws = workspace(c, device)
    return (_ptr(ws), 0 if ws is None else ws.numel() * ws.element_size())


# --------------------------------------------------------------------- TopK
def topk_compress(x: torch.Tensor, k: int, n_seg: int, ws=None, out: TopkPayload = None, blk: bool = True):
    """TopK per segment of x viewed as [n_seg, seg_len] -> TopkPayload"""
    L = _segments(x, n_seg)
    c = codec(TC_TOPK, n_seg, L, k, wire=_dt(x))
    if out is not None:
        _check_topk_payload(out, n_seg, k, L, x.dtype, x.device, "out")
    _need_gpu(x)
    if out is None:
        out = empty_topk_payload(n_seg, L, k, x.dtype, x.device, blk)
    p = Payload(_ptr(out.idx), _ptr(out.val), None, None, _ptr(out.blk))
    w, wn = _ws_args(c, x.device, ws)
    _check(lib().tc_topk_compress(C.byref(c), _ptr(x), _dt(x), C.byref(p), w, wn, _stream(x.device)),
           "tc_topk_compress")
    return out


def topk_decompress(pl: TopkPayload, seg_len: int, out_dtype=None, use_blk: bool = True, out: torch.Tensor = None):
    """dense [n_seg, seg_len] tensor: the sent values at their indices, +0 elsewhere"""
    if pl.idx.dim() != 2:
        raise ValueError("idx must be [n_seg, k]")
    n_seg, k = pl.idx.shape
    _check_topk_payload(pl, n_seg, k, seg_len, pl.val.dtype, pl.idx.device, "payload")
    if out is not None:
        if out.numel() != n_seg * seg_len:
            raise ValueError("out has the wrong element count")
        out_dtype = out.dtype
    out_dtype = out_dtype or pl.val.dtype
    _need_gpu(pl.idx, pl.val, pl.blk, out)
    c = codec(TC_TOPK, n_seg, seg_len, k, wire=_dt(pl.val))
    y = out if out is not None else torch.empty((n_seg, seg_len), dtype=out_dtype, device=pl.idx.device)
    p = Payload(_ptr(pl.idx), _ptr(pl.val), None, None, _ptr(pl.blk) if use_blk else None)
    _check(lib().tc_topk_decompress(C.byref(c), C.byref(p), _ptr(y), _DT[out_dtype], _stream(pl.idx.device)),
           "tc_topk_decompress")
    return y


def topk_gather(pl: TopkPayload, x: torch.Tensor, e: torch.Tensor = None, use_blk: bool = True,
                out: torch.Tensor = None) -> torch.Tensor:
    """x viewed as [n_seg, seg_len] at the indices of another tensor's TopK payload
    (the values sent in x's dtype); with e (float32, updated in place), X = x + e is
    sent and e <- X - received.  The receiver is topk_decompress(pl._replace(val=...))."""
    if pl.idx.dim() != 2:
        raise ValueError("idx must be [n_seg, k]")
    n_seg, k = pl.idx.shape
    L = _segments(x, n_seg)
    _check_topk_payload(pl, n_seg, k, L, x.dtype, x.device, "payload", need_val=False)
    if e is not None and (e.dtype != torch.float32 or e.numel() != x.numel()):
        raise ValueError("e must be float32 with x's element count")
    if out is not None and (tuple(out.shape) != (n_seg, k) or out.dtype != x.dtype):
        raise ValueError(f"out must be {x.dtype} [{n_seg}, {k}]")
    _need_gpu(pl.idx, pl.blk, x, e, out)
    val = out if out is not None else torch.empty((n_seg, k), dtype=x.dtype, device=x.device)
    c = codec(TC_TOPK, n_seg, L, k, wire=_dt(x))
    p = Payload(_ptr(pl.idx), None, None, None, _ptr(pl.blk) if use_blk else None)
    ep = None if e is None else C.cast(e.data_ptr(), C.POINTER(C.c_float))
    _check(lib().tc_topk_gather(C.byref(c), C.byref(p), _ptr(x), _dt(x), ep, _ptr(val), _stream(x.device)),
           "tc_topk_gather")
    return val


# ------------------------------------------------------------- quantization
def quant_pack(x: torch.Tensor, bits: int, n_grp: int, ws=None):
    """min-max quantization per group -> (codes uint8 [n_grp, group_bytes], meta f32 [n_grp, 2])"""
    _need_gpu(x)
    G = _segments(x, n_grp)
    c = codec(TC_QUANT, n_grp, G, bits=bits, wire=_dt(x))
    codes = torch.empty((n_grp, quant_group_bytes(G, bits)), dtype=torch.uint8, device=x.device)
    meta = torch.empty((n_grp, 2), dtype=torch.float32, device=x.device)
    p = Payload(None, None, _ptr(codes), _ptr(meta), None)
    w, wn = _ws_args(c, x.device, ws)
    _check(lib().tc_quant_pack(C.byref(c), _ptr(x), _dt(x), C.byref(p), w, wn, _stream(x.device)), "tc_quant_pack")
    return codes, meta


def quant_unpack(codes: torch.Tensor, meta: torch.Tensor, grp_len: int, bits: int, out_dtype=torch.float32,
                 out: torch.Tensor = None):
    """dense [n_grp, grp_len]: lo + code * scale per group"""
    n_grp = meta.shape[0]
    if meta.numel() != 2 * n_grp or meta.dtype != torch.float32:
        raise ValueError("meta must be float32 [n_grp, 2]")
    if codes.numel() != n_grp * quant_group_bytes(grp_len, bits):
        raise ValueError("codes have the wrong byte count for this group length and width")
    if out is not None:
        if out.numel() != n_grp * grp_len:
            raise ValueError("out has the wrong element count")
        out_dtype = out.dtype
    _need_gpu(codes, meta, out)
    c = codec(TC_QUANT, n_grp, grp_len, bits=bits, wire=_DT[out_dtype])
    y = out if out is not None else torch.empty((n_grp, grp_len), dtype=out_dtype, device=codes.device)
    p = Payload(None, None, _ptr(codes), _ptr(meta), None)
    _check(lib().tc_quant_unpack(C.byref(c), C.byref(p), _ptr(y), _DT[out_dtype], _stream(codes.device)),
           "tc_quant_unpack")
    return y


# ----------------------------------------------------------- error feedback
def ef_step_topk(x: torch.Tensor, e: torch.Tensor, k: int, n_seg: int, ws=None, out: TopkPayload = None,
                 blk: bool = True):
    """X = x + e; send TopK(X); e <- X - received.  e (float32) is updated in place."""
    if e.dtype != torch.float32 or e.numel() != x.numel():
        raise ValueError("e must be float32 with x's element count")
    L = _segments(x, n_seg)
    c = codec(TC_TOPK, n_seg, L, k, wire=_dt(x))
    if out is not None:
        _check_topk_payload(out, n_seg, k, L, x.dtype, x.device, "out")
    _need_gpu(x, e)
    if out is None:
        out = empty_topk_payload(n_seg, L, k, x.dtype, x.device, blk)
    p = Payload(_ptr(out.idx), _ptr(out.val), None, None, _ptr(out.blk))
    w, wn = _ws_args(c, x.device, ws)
    _check(lib().tc_ef_step(C.byref(c), _ptr(x), _dt(x), C.cast(e.data_ptr(), C.POINTER(C.c_float)), C.byref(p),
                            w, wn, _stream(x.device)), "tc_ef_step")
    return out


def ef_step_quant(x: torch.Tensor, e: torch.Tensor, bits: int, n_grp: int, ws=None, out=None):
    """X = x + e; send Q(X); e <- X - received.  e (float32) is updated in place.
    out: optional (codes, meta) to write into."""
    _need_gpu(x, e)
    if e.dtype != torch.float32 or e.numel() != x.numel():
        raise ValueError("e must be float32 with x's element count")
    G = _segments(x, n_grp)
    c = codec(TC_QUANT, n_grp, G, bits=bits, wire=_dt(x))
    if out is not None:
        codes, meta = out
        _need_gpu(codes, meta)
        if codes.numel() != n_grp * quant_group_bytes(G, bits) or meta.numel() != 2 * n_grp:
            raise ValueError("codes / meta have the wrong size")
    else:
        codes = torch.empty((n_grp, quant_group_bytes(G, bits)), dtype=torch.uint8, device=x.device)
        meta = torch.empty((n_grp, 2), dtype=torch.float32, device=x.device)
    p = Payload(None, None, _ptr(codes), _ptr(meta), None)
    w, wn = _ws_args(c, x.device, ws)
    _check(lib().tc_ef_step(C.byref(c), _ptr(x), _dt(x), C.cast(e.data_ptr(), C.POINTER(C.c_float)), C.byref(p),
                            w, wn, _stream(x.device)), "tc_ef_step")
    return codes, meta


class TopkQuantPayload(NamedTuple):
    """a TopK message whose kept values travel as b-bit min-max codes (one
    group per segment): indices, codes (uint8 [n_seg, group_bytes]), meta
    (float32 [n_seg, 2] = lo, scale) and the block table (or None)"""
    idx: torch.Tensor
    codes: torch.Tensor
    meta: torch.Tensor
    blk: Optional[torch.Tensor]
    bits: int


def empty_topk_quant_payload(n_seg: int, seg_len: int, k: int, bits: int, device,
                             blk: bool = True) -> TopkQuantPayload:
    return TopkQuantPayload(torch.empty((n_seg, k), dtype=torch.int32, device=device),
                            torch.empty((n_seg, quant_group_bytes(k, bits)), dtype=torch.uint8, device=device),
                            torch.empty((n_seg, 2), dtype=torch.float32, device=device),
                            torch.empty((n_seg, n_blocks(seg_len) + 1), dtype=torch.int32, device=device)
                            if blk else None,
                            bits)


def _check_topk_quant_payload(pl, n_seg: int, k: int, seg_len: int, bits: int, device, what: str):
    if pl.bits != bits:
        raise ValueError(f"{what} was made for {pl.bits} bits, not {bits}")
    _check_topk_payload(TopkPayload(pl.idx, None, pl.blk), n_seg, k, seg_len, None, device, what, need_val=False)
    if tuple(pl.codes.shape) != (n_seg, quant_group_bytes(k, bits)) or pl.codes.dtype != torch.uint8:
        raise ValueError(f"{what}.codes must be uint8 [{n_seg}, {quant_group_bytes(k, bits)}]")
    if tuple(pl.meta.shape) != (n_seg, 2) or pl.meta.dtype != torch.float32:
        raise ValueError(f"{what}.meta must be float32 [{n_seg}, 2]")
    for t in (pl.codes, pl.meta):
        if t.device != device or not t.is_contiguous():
            raise ValueError(f"{what} tensors must be contiguous on {device}")


def ef_step_topk_quant(x: torch.Tensor, e: torch.Tensor, k: int, bits: int, n_seg: int = 1, ws=None,
                       out: TopkQuantPayload = None, blk: bool = True) -> TopkQuantPayload:
    """X = x + e; send TopK(X) with the kept values quantized; e <- X - received
    (the receiver rounds to x's dtype).  e (float32) is updated in place."""
    if e.dtype != torch.float32 or e.numel() != x.numel():
        raise ValueError("e must be float32 with x's element count")
    L = _segments(x, n_seg)
    c = codec(TC_TOPK_QUANT, n_seg, L, k, bits=bits, wire=_dt(x))
    dev = x.device
    if out is not None:
        _check_topk_quant_payload(out, n_seg, k, L, bits, dev, "out")
    _need_gpu(x, e)
    if out is None:
        out = empty_topk_quant_payload(n_seg, L, k, bits, dev, blk)
    p = Payload(_ptr(out.idx), None, _ptr(out.codes), _ptr(out.meta), _ptr(out.blk))
    w, wn = _ws_args(c, dev, ws)
    _check(lib().tc_ef_step(C.byref(c), _ptr(x), _dt(x), C.cast(e.data_ptr(), C.POINTER(C.c_float)), C.byref(p),
                            w, wn, _stream(dev)), "tc_ef_step")
    return out


def topk_quant_decompress(pl: TopkQuantPayload, seg_len: int, out_dtype=torch.float32, use_blk: bool = True,
                          out: torch.Tensor = None):
    """dense [n_seg, seg_len]: lo + code * scale at the indices, +0 elsewhere"""
    if pl.idx.dim() != 2:
        raise ValueError("idx must be [n_seg, k]")
    n_seg, k = pl.idx.shape
    _check_topk_quant_payload(pl, n_seg, k, seg_len, pl.bits, pl.idx.device, "payload")
    if out is not None:
        if out.numel() != n_seg * seg_len:
            raise ValueError("out has the wrong element count")
        out_dtype = out.dtype
    _need_gpu(pl.idx, pl.codes, pl.meta, pl.blk, out)
    c = codec(TC_TOPK_QUANT, n_seg, seg_len, k, bits=pl.bits, wire=_DT[out_dtype])
    y = out if out is not None else torch.empty((n_seg, seg_len), dtype=out_dtype, device=pl.idx.device)
    p = Payload(_ptr(pl.idx), None, _ptr(pl.codes), _ptr(pl.meta), _ptr(pl.blk) if use_blk else None)
    _check(lib().tc_topk_decompress(C.byref(c), C.byref(p), _ptr(y), _DT[out_dtype], _stream(pl.idx.device)),
           "tc_topk_decompress")
    return y


# ----------------------------------------------------------------- EF-mixed
def efmix_counts(k: int) -> tuple:
    """(k_x, k_e): the input's and the error buffer's share of a budget of k
    (tc_efmix_counts)"""
    kx, ke = C.c_uint64(0), C.c_uint64(0)
    lib().tc_efmix_counts(k, C.byref(kx), C.byref(ke))
    return int(kx.value), int(ke.value)


def efmix_step(x: torch.Tensor, e: torch.Tensor, k: int, n_seg: int, out=None, blk: bool = True):
    """EF-mixed sender: TopK of x (k_x) and of e (k_e), both sent; e (float32,
    updated in place) keeps what was not sent.  Returns (payload_x, payload_e)."""
    if e.dtype != torch.float32 or e.numel() != x.numel():
        raise ValueError("e must be float32 with x's element count")
    L = _segments(x, n_seg)
    kx, ke = efmix_counts(k)
    c = codec(TC_TOPK, n_seg, L, k, wire=_dt(x))
    if out is not None:
        _check_topk_payload(out[0], n_seg, kx, L, x.dtype, x.device, "out[0]")
        _check_topk_payload(out[1], n_seg, ke, L, x.dtype, x.device, "out[1]")
    _need_gpu(x, e)
    if out is None:
        out = (empty_topk_payload(n_seg, L, kx, x.dtype, x.device, blk),
               empty_topk_payload(n_seg, L, ke, x.dtype, x.device, blk))
    px, pe = out
    a = Payload(_ptr(px.idx), _ptr(px.val), None, None, _ptr(px.blk))
    b = Payload(_ptr(pe.idx), _ptr(pe.val), None, None, _ptr(pe.blk))
    _check(lib().tc_efmix_step(C.byref(c), _ptr(x), _dt(x), C.cast(e.data_ptr(), C.POINTER(C.c_float)),
                               C.byref(a), C.byref(b), _stream(x.device)), "tc_efmix_step")
    return out


def efmix_reconstruct(px: TopkPayload, pe: TopkPayload, seg_len: int, out_dtype=None, use_blk: bool = True,
                      out: torch.Tensor = None):
    """dense [n_seg, seg_len]: the input's list written, the buffer's list added"""
    if px.idx.dim() != 2 or pe.idx.dim() != 2:
        raise ValueError("idx must be [n_seg, k]")
    n_seg, kx = px.idx.shape
    ke = pe.idx.shape[1]
    if pe.idx.shape[0] != n_seg or (kx, ke) != efmix_counts(kx + ke):
        raise ValueError("the two lists do not come from one EF-mixed budget")
    _check_topk_payload(px, n_seg, kx, seg_len, px.val.dtype, px.idx.device, "payload_x")
    _check_topk_payload(pe, n_seg, ke, seg_len, px.val.dtype, px.idx.device, "payload_e")
    if out is not None:
        if out.numel() != n_seg * seg_len:
            raise ValueError("out has the wrong element count")
        out_dtype = out.dtype
    out_dtype = out_dtype or px.val.dtype
    _need_gpu(px.idx, px.val, pe.idx, pe.val, out)
    c = codec(TC_TOPK, n_seg, seg_len, kx + ke, wire=_dt(px.val))
    y = out if out is not None else torch.empty((n_seg, seg_len), dtype=out_dtype, device=px.idx.device)
    a = Payload(_ptr(px.idx), _ptr(px.val), None, None, _ptr(px.blk) if use_blk else None)
    b = Payload(_ptr(pe.idx), _ptr(pe.val), None, None, _ptr(pe.blk) if use_blk else None)
    _check(lib().tc_efmix_reconstruct(C.byref(c), C.byref(a), C.byref(b), _ptr(y), _DT[out_dtype],
                                      _stream(px.idx.device)), "tc_efmix_reconstruct")
    return y


# ------------------------------------------------------------------- AQ-SGD
def _aqsgd_prepare(a, m, ids, k, out, blk):
    """shape checks of the AQ-SGD sender; returns (codec, n_ids, out, Payload)"""
    if ids.dtype != torch.int64 or a.dtype != m.dtype:
        raise TypeError("ids must be int64 and a, m share a dtype")
    if m.dim() != 2:
        raise ValueError("m must be [n_samples, seg_len]")
    if ids.dim() != 1:
        raise ValueError("ids must be one-dimensional")
    n_ids = ids.numel()
    L = m.shape[1]
    if a.numel() != n_ids * L:
        raise ValueError(f"a must hold n_ids * seg_len = {n_ids} * {L} elements")
    c = codec(TC_TOPK, n_ids, L, k, wire=_dt(m))
    if out is not None:
        _check_topk_payload(out, n_ids, k, L, a.dtype, a.device, "out")
    _need_gpu(a, m, ids)
    if out is None:
        out = empty_topk_payload(n_ids, L, k, a.dtype, a.device, blk)
    return c, n_ids, out, Payload(_ptr(out.idx), _ptr(out.val), None, None, _ptr(out.blk))


def aqsgd_step(a: torch.Tensor, m: torch.Tensor, ids: torch.Tensor, k: int, ws=None, out: TopkPayload = None,
               blk: bool = True):
    """sender: d = a - m[ids]; send TopK(d); m[ids] += sent.  m is updated in place."""
    c, n_ids, out, p = _aqsgd_prepare(a, m, ids, k, out, blk)
    w, wn = _ws_args(c, a.device, ws)
    _check(lib().tc_aqsgd_step(C.byref(c), _ptr(a), _dt(a), _ptr(m), m.shape[0], _ptr(ids), n_ids, C.byref(p),
                               w, wn, _stream(a.device)), "tc_aqsgd_step")
    return out


NOALLOC_SCRATCH_BYTES = 4 << 20   # TC_NOALLOC_SCRATCH_BYTES


def aqsgd_step_noalloc(a: torch.Tensor, m: torch.Tensor, ids: torch.Tensor, k: int, out: TopkPayload = None,
                       blk: bool = True):
    """aqsgd_step through the entry point that allocates nothing (its scratch is
    the library's own, shared by every call on the device); pass `out` to keep
    this call free of allocations on the Python side too."""
    c, n_ids, out, p = _aqsgd_prepare(a, m, ids, k, out, blk)
    _check(lib().tc_aqsgd_step_noalloc(C.byref(c), _ptr(a), _dt(a), _ptr(m), m.shape[0], _ptr(ids), n_ids,
                                       C.byref(p), _stream(a.device)), "tc_aqsgd_step_noalloc")
    return out


_ROW_IDS = {}


def _row_ids(n: int, device) -> torch.Tensor:
    """ids 0..n-1 on device (kept, so that a captured graph holds no allocation)"""
    key = (n, str(device))
    t = _ROW_IDS.get(key)
    if t is None:
        t = _ROW_IDS[key] = torch.arange(n, dtype=torch.int64, device=device)
    return t


def ef21_step(x: torch.Tensor, g: torch.Tensor, k: int, ws=None, out: TopkPayload = None, blk: bool = True):
    """EF21 sender (Sec. 2.4): send C(x - g) with C = TopK, then g <- g + C(x - g);
    x and g are [n_seg, seg_len] of one dtype, g (the previously sent value) is
    updated in place.  This is the Sec. 2.5 AQ-SGD sender with one buffer row
    per segment (ids 0..n_seg-1)."""
    return aqsgd_step(x, g, _row_ids(g.shape[0], g.device), k, ws=ws, out=out, blk=blk)


def ef21_reconstruct(pl: TopkPayload, g_r: torch.Tensor, out=None, use_blk: bool = True):
    """EF21 receiver: g_r <- g_r + received; returns g_r (a copy in `out` if given)"""
    return aqsgd_reconstruct(pl, g_r, _row_ids(g_r.shape[0], g_r.device), out=out, use_blk=use_blk)


def aqsgd_reconstruct(pl: TopkPayload, m_r: torch.Tensor, ids: torch.Tensor, out=None, use_blk: bool = True):
    """receiver: m_r[ids] += received; returns a_hat = m_r[ids].  m_r is updated in place."""
    if ids.dtype != torch.int64 or ids.dim() != 1:
        raise TypeError("ids must be one-dimensional int64")
    if m_r.dim() != 2:
        raise ValueError("m_r must be [n_samples, seg_len]")
    if pl.idx.dim() != 2:
        raise ValueError("idx must be [n_ids, k]")
    n_ids, k = pl.idx.shape
    L = m_r.shape[1]
    if ids.numel() != n_ids:
        raise ValueError(f"the payload has {n_ids} segments, ids {ids.numel()}")
    _check_topk_payload(pl, n_ids, k, L, m_r.dtype, m_r.device, "payload")
    if out is not None and (out.numel() != n_ids * L or out.dtype != m_r.dtype):
        raise ValueError(f"out must be {m_r.dtype} with {n_ids} * {L} elements")
    _need_gpu(pl.idx, pl.val, pl.blk, m_r, ids, out)
    c = codec(TC_TOPK, n_ids, L, k, wire=_dt(m_r))
    a_hat = torch.empty((n_ids, L), dtype=m_r.dtype, device=m_r.device) if out is None else out
    p = Payload(_ptr(pl.idx), _ptr(pl.val), None, None, _ptr(pl.blk) if use_blk else None)
    _check(lib().tc_aqsgd_reconstruct(C.byref(c), C.byref(p), _ptr(m_r), _dt(m_r), m_r.shape[0], _ptr(ids), n_ids,
                                      _ptr(a_hat), _stream(m_r.device)), "tc_aqsgd_reconstruct")
    return a_hat
