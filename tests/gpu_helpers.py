"""Shared helpers of the GPU parity tests: raw views of torch tensors for the
oracle (which takes binary16/bfloat16 as uint16 patterns), and comparisons."""
import numpy as np
import torch

DTN = {torch.float32: "f32", torch.bfloat16: "bf16", torch.float16: "f16"}
TORCH = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}


def raw(t: torch.Tensor) -> np.ndarray:
    """torch tensor -> numpy array of its elements' raw patterns (float32 stays float32)"""
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.float32:
        return t.numpy()
    if t.dtype in (torch.bfloat16, torch.float16):
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.int32:
        return t.numpy().view(np.uint32)
    return t.numpy()


def from_raw(a: np.ndarray, dt: str, device) -> torch.Tensor:
    if dt == "f32":
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(device)
    t = torch.from_numpy(np.ascontiguousarray(a, np.uint16).view(np.int16))
    return t.view(TORCH[dt]).to(device)


def bits(a: np.ndarray) -> np.ndarray:
    """bit patterns for exact comparison (float32 -> uint32)"""
    a = np.ascontiguousarray(a)
    return a.view(np.uint32) if a.dtype == np.float32 else a


def assert_bits_equal(got, want, what):
    g, w = bits(got), bits(want)
    assert g.shape == w.shape, f"{what}: shape {g.shape} != {w.shape}"
    bad = np.flatnonzero(g.ravel() != w.ravel())
    assert bad.size == 0, (f"{what}: {bad.size} of {g.size} differ; first at {bad[:5].tolist()}: "
                           f"got {g.ravel()[bad[:5]].tolist()} want {w.ravel()[bad[:5]].tolist()}")


def assert_rel_close(got, want, rel, what):
    """binary32 buffers within `rel` relative (exact zeros must match exactly)"""
    g = np.asarray(got, np.float64).ravel()
    w = np.asarray(want, np.float64).ravel()
    err = np.abs(g - w)
    lim = rel * np.abs(w)
    bad = np.flatnonzero(err > lim)
    assert bad.size == 0, f"{what}: {bad.size} entries beyond {rel} relative; first {bad[:5].tolist()}"


def check_block_table(blk, oracle_idx, L, what="blk"):
    """blk[s][b] must count the kept indices below b * 4096 (and end with k)"""
    g = raw(blk).astype(np.int64)
    n_seg, k = oracle_idx.shape
    nb = (L + 4095) // 4096
    assert g.shape == (n_seg, nb + 1), f"{what}: shape {g.shape}"
    bounds = np.arange(nb + 1, dtype=np.int64) * 4096
    for s in range(n_seg):
        want = np.searchsorted(oracle_idx[s].astype(np.int64), bounds, side="left")
        want[-1] = k
        assert np.array_equal(g[s], want), f"{what}: segment {s}: got {g[s][:8]} want {want[:8]}"
