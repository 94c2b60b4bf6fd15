"""Pins for the oracle's format conversions (binary32 <-> binary16 / bfloat16).

Checked against: IEEE halfway cases worked by hand (tests/golden/conv_halfway.txt),
exhaustive round trips, numpy's float16 cast and torch's CPU bfloat16 cast
(both round to nearest even).
"""
import numpy as np
import pytest
import torch

from conftest import read_golden


def _f32_from_hex(h):
    return np.array([int(h, 16)], np.uint32).view(np.float32)


def test_halfway_cases(orc):
    g = read_golden("conv_halfway.txt")
    for src, want in g["bf16"]:
        got = orc.from_f32(_f32_from_hex(src), "bf16")[0]
        assert got == int(want, 16), (src, hex(got), want)
    for src, want in g["f16"]:
        got = orc.from_f32(_f32_from_hex(src), "f16")[0]
        assert got == int(want, 16), (src, hex(got), want)


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_exhaustive_round_trip(orc, dt):
    pats = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    f = orc.to_f32(pats, dt)
    back = orc.from_f32(f, dt)
    if dt == "bf16":
        nan = ((pats & 0x7F80) == 0x7F80) & ((pats & 0x007F) != 0)
    else:
        nan = ((pats & 0x7C00) == 0x7C00) & ((pats & 0x03FF) != 0)
    assert np.isnan(f[nan]).all()
    assert (back[~nan] == pats[~nan]).all()


def test_f16_upcast_matches_numpy(orc):
    pats = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = pats.view(np.float16).astype(np.float32)
    got = orc.to_f32(pats, "f16")
    fin = np.isfinite(ref)
    assert (got[fin].view(np.uint32) == ref[fin].view(np.uint32)).all()


def _probe_floats(n=200_000, seed=1):
    rng = np.random.default_rng(seed)
    bits = rng.integers(0, 2**32, size=n, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    # plus values near binary16 range edges, its subnormals and exact midpoints
    near = (rng.standard_normal(n).astype(np.float32) * np.float32(2.0) **
            rng.integers(-30, 17, size=n).astype(np.float32))
    mids = (np.arange(0, 65536, dtype=np.uint32).astype(np.uint16).view(np.float16).astype(np.float64))
    mids = mids[np.isfinite(mids)]
    mid = ((mids[:-1] + mids[1:]) / 2).astype(np.float32)      # exact in binary32
    out = np.concatenate([x, near, mid])
    return out[np.isfinite(out)]


def test_f16_downcast_matches_numpy(orc):
    x = _probe_floats()
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    got = orc.from_f32(x, "f16")
    assert (got == ref).all()


def test_bf16_downcast_matches_torch(orc):
    x = _probe_floats(seed=2)
    x = x[np.abs(x) < np.float32(3e38)]
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = orc.from_f32(x, "bf16")
    assert (got == ref).all()
    # subnormal binary32 inputs keep their subnormal bfloat16 image
    sub = np.array([1, 0x7FFF, 0x8000, 0x8001, 0x18000, 0x7FFFFF], np.uint32).view(np.float32)
    ref = torch.from_numpy(sub).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (orc.from_f32(sub, "bf16") == ref).all()
