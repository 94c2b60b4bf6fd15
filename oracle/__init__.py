"""The CPU oracle: a plain, slow implementation of the paper's compressors.

TEST INFRASTRUCTURE ONLY.  It is loaded by the test suite, by the smoke check
and by the CPU-baseline leg of the benchmark, never by the GPU library or its
binding.  It shares no code with the GPU path.

Arrays are numpy arrays.  Elements of dtype "f32" are float32; "bf16" and
"f16" elements are carried as their raw 16-bit patterns in uint16 arrays.
The arithmetic lives in ``tco.c``; this module only marshals arguments.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# TCO_LIB names another build of tco.c (the sanitized one of the test suite)
_LIB_PATH = os.environ.get("TCO_LIB") or os.path.join(_HERE, "liboracle.so")

DT = {"f32": 0, "bf16": 1, "f16": 2}
_NP = {"f32": np.float32, "bf16": np.uint16, "f16": np.uint16}

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        L = C.CDLL(_LIB_PATH)
        u64, u32, i32, vp = C.c_uint64, C.c_uint32, C.c_int, C.c_void_p
        sig = {
            "tco_f16_to_f32": (C.c_float, [C.c_uint16]),
            "tco_f32_to_f16": (C.c_uint16, [C.c_float]),
            "tco_bf16_to_f32": (C.c_float, [C.c_uint16]),
            "tco_f32_to_bf16": (C.c_uint16, [C.c_float]),
            "tco_topk_count": (u64, [u64, u32, u32]),
            "tco_topk_indices": (i32, [vp, u64, u64, vp]),
            "tco_topk_compress": (i32, [vp, i32, u64, u64, u64, i32, vp, vp, i32]),
            "tco_topk_decompress": (i32, [vp, vp, i32, u64, u64, u64, vp, i32]),
            "tco_topk_gather": (i32, [vp, i32, vp, u64, u64, u64, vp, i32, vp]),
            "tco_quant_group_bytes": (u64, [u64, u32]),
            "tco_quant_group": (i32, [vp, u64, u32, vp, vp]),
            "tco_quant_pack": (i32, [vp, i32, u64, u64, u32, vp, vp, i32]),
            "tco_quant_unpack": (i32, [vp, vp, u64, u64, u32, vp, i32]),
            "tco_ef_topk": (i32, [vp, i32, vp, u64, u64, u64, i32, vp, vp, i32]),
            "tco_ef_quant": (i32, [vp, i32, vp, u64, u64, u32, i32, vp, vp, i32]),
            "tco_ef_topk_quant": (i32, [vp, i32, vp, u64, u64, u64, u32, i32, vp, vp, vp, i32]),
            "tco_topk_quant_decompress": (i32, [vp, vp, vp, u64, u64, u64, u32, vp, i32]),
            "tco_aqsgd_send": (i32, [vp, vp, i32, u64, u64, vp, u64, u64, vp, vp, i32]),
            "tco_aqsgd_recv": (i32, [vp, vp, vp, i32, u64, u64, vp, u64, u64, vp]),
            "tco_efmix_kx": (u64, [u64]),
            "tco_efmix_ke": (u64, [u64]),
            "tco_efmix_send": (i32, [vp, i32, vp, u64, u64, u64, vp, vp, vp, vp]),
            "tco_efmix_recv": (i32, [vp, vp, vp, vp, i32, u64, u64, u64, vp, i32]),
            "tco_to_f32": (None, [vp, i32, u64, vp]),
            "tco_from_f32": (None, [vp, u64, i32, vp]),
            "tco_through": (C.c_float, [i32, C.c_float]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(C.c_void_p)


def _chk(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments")


def _raw(x: np.ndarray, dt: str) -> np.ndarray:
    x = np.ascontiguousarray(x)
    want = _NP[dt]
    if x.dtype != want:
        raise TypeError(f"dtype {dt} needs a {np.dtype(want).name} array, got {x.dtype}")
    return x


# ---------------------------------------------------------------- conversions
def to_f32(x: np.ndarray, dt: str) -> np.ndarray:
    """exact upcast of raw elements of dtype dt to float32"""
    x = _raw(x, dt)
    out = np.empty(x.shape, np.float32)
    lib().tco_to_f32(_p(x), DT[dt], x.size, _p(out))
    return out


def from_f32(x: np.ndarray, dt: str) -> np.ndarray:
    """round-to-nearest-even downcast of float32 to dtype dt (raw elements)"""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, _NP[dt])
    lib().tco_from_f32(_p(x), x.size, DT[dt], _p(out))
    return out


# ----------------------------------------------------------------------- TopK
def topk_count(L: int, num: int, den: int) -> int:
    return int(lib().tco_topk_count(L, num, den))


def topk_indices(v: np.ndarray, k: int) -> np.ndarray:
    v = np.ascontiguousarray(v, dtype=np.float32).ravel()
    idx = np.zeros(max(k, 1), np.uint32)
    _chk(lib().tco_topk_indices(_p(v), v.size, k, _p(idx)), "topk_indices")
    return idx[:k].copy()


def topk_compress(x, dt, n_seg, L, k, wire=None, threads=0):
    wire = wire or dt
    x = _raw(x, dt)
    assert x.size == n_seg * L
    idx = np.zeros((n_seg, k), np.uint32)
    val = np.zeros((n_seg, k), _NP[wire])
    _chk(lib().tco_topk_compress(_p(x), DT[dt], n_seg, L, k, DT[wire], _p(idx), _p(val), threads),
         "topk_compress")
    return idx, val


def topk_decompress(idx, val, wire, n_seg, L, k, out_dt=None):
    out_dt = out_dt or wire
    idx = np.ascontiguousarray(idx, np.uint32)
    val = _raw(val, wire)
    y = np.zeros((n_seg, L), _NP[out_dt])
    _chk(lib().tco_topk_decompress(_p(idx), _p(val), DT[wire], n_seg, L, k, _p(y), DT[out_dt]),
         "topk_decompress")
    return y


def topk_gather(x, dt, idx, n_seg, L, k, e=None, wire=None):
    """TopK at given indices (Sec. 3.2: gradients compressed at the indices
    the activations' TopK kept): returns val, or (val, e_next) when e is given
    (error feedback around this compressor); e is not modified"""
    wire = wire or dt
    x = _raw(x, dt)
    assert x.size == n_seg * L
    idx = np.ascontiguousarray(idx, np.uint32)
    assert idx.size == n_seg * k
    val = np.zeros((n_seg, k), _NP[wire])
    e2 = None if e is None else np.array(e, dtype=np.float32, copy=True, order="C")
    _chk(lib().tco_topk_gather(_p(x), DT[dt], None if e2 is None else _p(e2), n_seg, L, k, _p(idx), DT[wire],
                               _p(val)), "topk_gather")
    return val if e is None else (val, e2)


# --------------------------------------------------------------- quantization
def quant_group_bytes(G: int, b: int) -> int:
    return 4 * G if b == 32 else int(lib().tco_quant_group_bytes(G, b))


def quant_pack(x, dt, n_grp, G, b, threads=0):
    x = _raw(x, dt)
    assert x.size == n_grp * G
    codes = np.zeros((n_grp, quant_group_bytes(G, b)), np.uint8)
    meta = np.zeros((n_grp, 2), np.float32)
    _chk(lib().tco_quant_pack(_p(x), DT[dt], n_grp, G, b, _p(codes), _p(meta), threads), "quant_pack")
    return codes, meta


def quant_unpack(codes, meta, n_grp, G, b, out_dt="f32"):
    codes = np.ascontiguousarray(codes, np.uint8)
    meta = np.ascontiguousarray(meta, np.float32)
    y = np.zeros((n_grp, G), _NP[out_dt])
    _chk(lib().tco_quant_unpack(_p(codes), _p(meta), n_grp, G, b, _p(y), DT[out_dt]), "quant_unpack")
    return y


# ------------------------------------------------------------- error feedback
def ef_topk(x, dt, e, n_seg, L, k, wire=None, threads=0):
    """returns (idx, val, e_next); e is not modified"""
    wire = wire or dt
    x = _raw(x, dt)
    e2 = np.array(e, dtype=np.float32, copy=True, order="C")
    idx = np.zeros((n_seg, k), np.uint32)
    val = np.zeros((n_seg, k), _NP[wire])
    _chk(lib().tco_ef_topk(_p(x), DT[dt], _p(e2), n_seg, L, k, DT[wire], _p(idx), _p(val), threads),
         "ef_topk")
    return idx, val, e2


def ef_quant(x, dt, e, n_grp, G, b, out_dt=None, threads=0):
    """returns (codes, meta, e_next); e is not modified"""
    out_dt = out_dt or dt
    x = _raw(x, dt)
    e2 = np.array(e, dtype=np.float32, copy=True, order="C")
    codes = np.zeros((n_grp, quant_group_bytes(G, b)), np.uint8)
    meta = np.zeros((n_grp, 2), np.float32)
    _chk(lib().tco_ef_quant(_p(x), DT[dt], _p(e2), n_grp, G, b, DT[out_dt], _p(codes), _p(meta), threads),
         "ef_quant")
    return codes, meta, e2


def ef_topk_quant(x, dt, e, n_seg, L, k, b, out_dt=None, threads=0):
    """returns (idx, codes, meta, e_next); e is not modified"""
    out_dt = out_dt or dt
    x = _raw(x, dt)
    e2 = np.array(e, dtype=np.float32, copy=True, order="C")
    idx = np.zeros((n_seg, k), np.uint32)
    codes = np.zeros((n_seg, quant_group_bytes(k, b)), np.uint8)
    meta = np.zeros((n_seg, 2), np.float32)
    _chk(lib().tco_ef_topk_quant(_p(x), DT[dt], _p(e2), n_seg, L, k, b, DT[out_dt], _p(idx), _p(codes),
                                 _p(meta), threads), "ef_topk_quant")
    return idx, codes, meta, e2


def topk_quant_decompress(idx, codes, meta, n_seg, L, k, b, out_dt):
    idx = np.ascontiguousarray(idx, np.uint32)
    codes = np.ascontiguousarray(codes, np.uint8)
    meta = np.ascontiguousarray(meta, np.float32)
    y = np.zeros((n_seg, L), _NP[out_dt])
    _chk(lib().tco_topk_quant_decompress(_p(idx), _p(codes), _p(meta), n_seg, L, k, b, _p(y), DT[out_dt]),
         "topk_quant_decompress")
    return y


# --------------------------------------------------------------------- AQ-SGD
def aqsgd_send(a, m, dt, ids, k, threads=0):
    """sender side; updates the buffer m [n_samples, L] in place; returns (idx, val)"""
    a = _raw(a, dt)
    assert m.flags["C_CONTIGUOUS"] and m.dtype == _NP[dt]
    n_samples, L = m.shape
    ids = np.ascontiguousarray(ids, np.int64)
    idx = np.zeros((ids.size, k), np.uint32)
    val = np.zeros((ids.size, k), _NP[dt])
    _chk(lib().tco_aqsgd_send(_p(a), _p(m), DT[dt], n_samples, L, _p(ids), ids.size, k, _p(idx), _p(val),
                              threads), "aqsgd_send")
    return idx, val


def aqsgd_recv(idx, val, m_r, dt, ids, k):
    """receiver side; updates m_r in place; returns a_hat [n_ids, L]"""
    assert m_r.flags["C_CONTIGUOUS"] and m_r.dtype == _NP[dt]
    n_samples, L = m_r.shape
    ids = np.ascontiguousarray(ids, np.int64)
    idx = np.ascontiguousarray(idx, np.uint32)
    val = _raw(val, dt)
    a_hat = np.zeros((ids.size, L), _NP[dt])
    _chk(lib().tco_aqsgd_recv(_p(idx), _p(val), _p(m_r), DT[dt], n_samples, L, _p(ids), ids.size, k,
                              _p(a_hat)), "aqsgd_recv")
    return a_hat


# ------------------------------------------------------------------ EF-mixed
def efmix_counts(k: int) -> tuple[int, int]:
    """(k_x, k_e): entries of the input and of the error buffer in a budget of k"""
    return int(lib().tco_efmix_kx(k)), int(lib().tco_efmix_ke(k))


def efmix_send(x, dt, e, n_seg, L, k):
    """returns (idx_x, val_x, idx_e, val_e, e_next); e is not modified"""
    kx, ke = efmix_counts(k)
    x = _raw(x, dt)
    e2 = np.array(e, dtype=np.float32, copy=True, order="C")
    idx_x = np.zeros((n_seg, kx), np.uint32)
    val_x = np.zeros((n_seg, kx), _NP[dt])
    idx_e = np.zeros((n_seg, ke), np.uint32)
    val_e = np.zeros((n_seg, ke), _NP[dt])
    _chk(lib().tco_efmix_send(_p(x), DT[dt], _p(e2), n_seg, L, k, _p(idx_x), _p(val_x), _p(idx_e), _p(val_e)),
         "efmix_send")
    return idx_x, val_x, idx_e, val_e, e2


def efmix_recv(idx_x, val_x, idx_e, val_e, wire, n_seg, L, k, out_dt="f32"):
    """the receiver's dense [n_seg, L] in out_dt"""
    idx_x = np.ascontiguousarray(idx_x, np.uint32)
    idx_e = np.ascontiguousarray(idx_e, np.uint32)
    val_x, val_e = _raw(val_x, wire), _raw(val_e, wire)
    y = np.zeros((n_seg, L), _NP[out_dt])
    _chk(lib().tco_efmix_recv(_p(idx_x), _p(val_x), _p(idx_e), _p(val_e), DT[wire], n_seg, L, k, _p(y),
                              DT[out_dt]), "efmix_recv")
    return y
