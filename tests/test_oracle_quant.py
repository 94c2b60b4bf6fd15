"""Pins for the oracle's uniform b-bit min-max quantization (Sec. 2.2: map the
vector onto [0,1] with min-max scaling, quantize to 2^b levels, decompress back
to the original scale; 2, 4, 6 and 8 bits are the studied widths).

Checked against: hand-worked examples (tests/golden/quant_w2_w5.txt), numpy's
bit packing (np.packbits, little bit order) as an independent packer, the exact
(binary64) level u*(2^b-1), the worst-case reconstruction error scale/2,
special cases (constant group, b = 32 pass-through, -0, subnormal ranges).
"""
import numpy as np
import pytest

from conftest import read_golden

G_ = read_golden("quant_w2_w5.txt")


def _bytes(hexes):
    return [int(h, 16) for h in hexes]


def _unpack_codes(stream, G, b):
    """independent decoder: numpy unpackbits, LSB-first"""
    bits = np.unpackbits(np.asarray(stream, np.uint8), bitorder="little")[: G * b]
    bits = bits.reshape(G, b).astype(np.uint32)
    return (bits << np.arange(b, dtype=np.uint32)).sum(axis=1)


def _pack_codes(codes, b, nbytes):
    bits = ((np.asarray(codes, np.uint32)[:, None] >> np.arange(b, dtype=np.uint32)) & 1).astype(np.uint8)
    out = np.packbits(bits.ravel(), bitorder="little")
    return np.concatenate([out, np.zeros(nbytes - out.size, np.uint8)])


@pytest.mark.parametrize("w", ["w2", "w3", "w5"])
def test_worked_codes(orc, w):
    v = np.array([float(t) for t in G_[f"{w}_v"]], np.float32)
    b = int(G_[f"{w}_b"][0])
    codes, meta = orc.quant_pack(v, "f32", 1, v.size, b)
    assert _unpack_codes(codes[0], v.size, b).tolist() == [int(t) for t in G_[f"{w}_codes"]]
    if f"{w}_bytes" in G_:
        assert codes[0].tolist() == _bytes(G_[f"{w}_bytes"])
    if f"{w}_lo" in G_:
        assert meta[0].tolist() == [float(G_[f"{w}_lo"][0]), float(G_[f"{w}_scale"][0])]


def test_worked_w4_bytes(orc):
    v = np.arange(16, dtype=np.float32)
    codes, meta = orc.quant_pack(v, "f32", 1, 16, 4)
    assert codes[0].tolist() == _bytes(G_["w4_bytes"])
    assert meta[0].tolist() == [0.0, 1.0]


def test_on_grid_is_exact(orc):
    v = (np.float32(-1) + np.arange(16, dtype=np.float32) / np.float32(8)).astype(np.float32)
    codes, meta = orc.quant_pack(v, "f32", 1, 16, 4)
    assert meta[0, 1] == float(G_["grid_scale"][0])
    assert _unpack_codes(codes[0], 16, 4).tolist() == list(range(16))
    y = orc.quant_unpack(codes, meta, 1, 16, 4)
    assert (y[0].view(np.uint32) == v.view(np.uint32)).all()


@pytest.mark.parametrize("b", [1, 2, 3, 4, 5, 6, 7, 8])
@pytest.mark.parametrize("G", [1, 5, 31, 32, 33, 100, 768, 1000])
def test_codes_levels_and_bound(orc, b, G):
    rng = np.random.default_rng(1000 * b + G)
    n_grp = 3
    x = (rng.standard_normal((n_grp, G)) * rng.choice([1e-3, 1.0, 50.0], size=(n_grp, 1))).astype(np.float32)
    codes, meta = orc.quant_pack(x, "f32", n_grp, G, b)
    gb = 4 * ((G * b + 31) // 32)
    assert codes.shape == (n_grp, gb)
    y = orc.quant_unpack(codes, meta, n_grp, G, b)
    L = (1 << b) - 1
    for g in range(n_grp):
        v = x[g].astype(np.float64)
        lo, hi = v.min(), v.max()
        c = _unpack_codes(codes[g], G, b)
        # the stream re-packs to the same bytes, padding bits included
        assert (_pack_codes(c, b, gb) == codes[g]).all()
        assert meta[g, 0] == np.float32(lo)
        if hi == lo:
            assert (c == 0).all() and meta[g, 1] == 0
            continue
        assert np.float32(meta[g, 1]) == np.float32(np.float32(hi - lo) / np.float32(L))
        # code is the nearest of the 2^b levels to u*(2^b-1), up to binary32 slop
        t = (v - lo) / (hi - lo) * L
        assert (np.abs(c - t) <= 0.5 + 1e-5 * L).all()
        assert c[v.argmin()] == 0 and c[v.argmax()] == L
        order = np.argsort(v, kind="stable")
        assert (np.diff(c[order].astype(np.int64)) >= 0).all()        # monotone in v
        # reconstruction error at most half a step (plus rounding of the decode)
        scale = float(meta[g, 1])
        ulp = np.spacing(np.float32(max(abs(lo), abs(hi)))).astype(np.float64)
        assert (np.abs(y[g].astype(np.float64) - v) <= scale / 2 + 2 * ulp).all()


def test_constant_group_and_negative_zero(orc):
    v = np.full(40, -0.0, np.float32)
    codes, meta = orc.quant_pack(v, "f32", 1, 40, 4)
    assert (codes == 0).all()
    assert meta[0].view(np.uint32).tolist() == [0, 0]           # lo canonicalized to +0
    v = np.full(40, 2.5, np.float32)
    codes, meta = orc.quant_pack(v, "f32", 1, 40, 4)
    y = orc.quant_unpack(codes, meta, 1, 40, 4)
    assert (codes == 0).all() and meta[0].tolist() == [2.5, 0.0] and (y == 2.5).all()
    # a -0 minimum reads as +0 in the metadata; the reconstruction is unaffected
    v = np.array([-0.0, 1.0, 0.5], np.float32)
    codes, meta = orc.quant_pack(v, "f32", 1, 3, 2)
    assert meta[0].view(np.uint32)[0] == 0


def test_subnormal_range_is_kept(orc):
    tiny = np.float32(2.0) ** -139
    v = np.array([0.0, tiny / 2, tiny], np.float32)
    codes, meta = orc.quant_pack(v, "f32", 1, 3, 1)
    assert meta[0, 1] == tiny                                  # no flush to zero
    assert _unpack_codes(codes[0], 3, 1).tolist() == [0, 0, 1]  # u = 0.5 ties to even
    y = orc.quant_unpack(codes, meta, 1, 3, 1)
    assert y[0].tolist() == [0.0, 0.0, float(tiny)]


def test_b32_is_identity(orc):
    rng = np.random.default_rng(4)
    x = rng.standard_normal((2, 77)).astype(np.float32)
    x[0, 3] = -0.0
    codes, meta = orc.quant_pack(x, "f32", 2, 77, 32)
    y = orc.quant_unpack(codes, meta, 2, 77, 32)
    assert (y.view(np.uint32) == x.view(np.uint32)).all()


def test_bf16_output_rounds_reconstruction(orc):
    rng = np.random.default_rng(9)
    x = orc.from_f32(rng.standard_normal((4, 768)).astype(np.float32), "bf16")
    codes, meta = orc.quant_pack(x, "bf16", 4, 768, 4)
    y32 = orc.quant_unpack(codes, meta, 4, 768, 4, "f32")
    y16 = orc.quant_unpack(codes, meta, 4, 768, 4, "bf16")
    assert (y16 == orc.from_f32(y32, "bf16")).all()
