"""Pins for the oracle's error feedback (Sec. 2.4: e = X - C(X), the next round
sends C(X + e); one global buffer per compression operator, added to the next
batch).

Checked against: the hand-worked example tests/golden/ef_w6.txt; exact
telescoping (sum of what the receiver got + final residual == sum of inputs)
on a dyadic grid where every binary32 add is exact; the per-step identity
r + e' == X; the K = 100% / K = 0 / b = 32 special cases; and for the
quantizer, telescoping within the binary32 rounding bound.
"""
import numpy as np
import pytest

from conftest import read_golden


def _vec(g, k):
    return np.array([float(t) for t in g[k]], np.float32)


def test_worked_example_w6(orc):
    g = read_golden("ef_w6.txt")
    e = np.zeros(3, np.float32)
    for step in (1, 2):
        idx, val, e = orc.ef_topk(_vec(g, f"x{step}"), "f32", e, 1, 3, 1)
        sent = orc.topk_decompress(idx, val, "f32", 1, 3, 1)[0]
        assert sent.tolist() == _vec(g, f"sent{step}").tolist()
        assert e.tolist() == _vec(g, f"e{step}").tolist()


def _dyadic(rng, shape, jmax):
    return (rng.integers(-jmax, jmax + 1, size=shape).astype(np.float32) / np.float32(256)).astype(np.float32)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("frac", [(0, 1), (1, 10), (3, 10), (1, 1)])
def test_topk_telescoping_exact(orc, dt, frac):
    rng = np.random.default_rng(17)
    n_seg, L, T = 4, 50, 64
    k = orc.topk_count(L, *frac)
    jmax = 2 ** 10 if dt == "f32" else 2 ** 7      # inputs exact in the input dtype
    e = np.zeros((n_seg, L), np.float32)
    tot_x = np.zeros((n_seg, L))
    tot_r = np.zeros((n_seg, L))
    for _ in range(T):
        x32 = _dyadic(rng, (n_seg, L), jmax)
        x = x32 if dt == "f32" else orc.from_f32(x32, "bf16")
        assert (orc.to_f32(x, dt) == x32).all()
        X = orc.to_f32(x, dt) + e                         # what the step compresses
        idx, val, e = orc.ef_topk(x, dt, e, n_seg, L, k)
        r = orc.to_f32(orc.topk_decompress(idx, val, dt, n_seg, L, k), dt)
        assert ((r + e).view(np.uint32) == X.view(np.uint32)).all()     # r + e' == X exactly
        tot_x += x32
        tot_r += r
    assert (tot_r + e == tot_x).all()
    if frac == (1, 1) and dt == "f32":
        assert (e == 0).all()
    if frac == (0, 1):
        assert (tot_r == 0).all() and (e == tot_x).all()


def test_topk_step_identity_random(orc):
    rng = np.random.default_rng(3)
    for dt in ("f32", "bf16", "f16"):
        x = rng.standard_normal((8, 1000)).astype(np.float32)
        x = x if dt == "f32" else orc.from_f32(x, dt)
        e = (rng.standard_normal((8, 1000)) * 0.1).astype(np.float32)
        X = orc.to_f32(x, dt) + e
        idx, val, e2 = orc.ef_topk(x, dt, e, 8, 1000, 100)
        r = orc.to_f32(orc.topk_decompress(idx, val, dt, 8, 1000, 100), dt)
        assert ((r + e2).view(np.uint32) == X.view(np.uint32)).all()
        # kept indices are the TopK of X itself
        for s in range(8):
            assert (idx[s] == orc.topk_indices(X[s], 100)).all()


@pytest.mark.parametrize("b", [2, 4, 8])
def test_quant_telescoping_within_rounding(orc, b):
    rng = np.random.default_rng(b)
    n_grp, G, T = 3, 256, 32
    e = np.zeros((n_grp, G), np.float32)
    tot_x = np.zeros((n_grp, G))
    tot_r = np.zeros((n_grp, G))
    slop = np.zeros((n_grp, G))
    for _ in range(T):
        x = rng.standard_normal((n_grp, G)).astype(np.float32)
        X = x + e
        codes, meta, e = orc.ef_quant(x, "f32", e, n_grp, G, b)
        r = orc.quant_unpack(codes, meta, n_grp, G, b)
        # the residual is what the receiver missed, up to one rounding of each op
        assert (np.abs((X.astype(np.float64) - r) - e) <= np.spacing(np.abs(e))).all()
        tot_x += x
        tot_r += r
        slop += np.spacing(np.abs(X)).astype(np.float64) + np.spacing(np.abs(e)).astype(np.float64)
    assert (np.abs(tot_r + e - tot_x) <= slop).all()


def test_quant_b32_leaves_no_residual(orc):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((2, 300)).astype(np.float32)
    e = (rng.standard_normal((2, 300)) * 0.01).astype(np.float32)
    codes, meta, e2 = orc.ef_quant(x, "f32", e, 2, 300, 32)
    assert (e2 == 0).all()


def test_bf16_quant_residual_uses_bf16_reconstruction(orc):
    rng = np.random.default_rng(8)
    x = orc.from_f32(rng.standard_normal((4, 768)).astype(np.float32), "bf16")
    e = (rng.standard_normal((4, 768)) * 0.01).astype(np.float32)
    X = orc.to_f32(x, "bf16") + e
    codes, meta, e2 = orc.ef_quant(x, "bf16", e, 4, 768, 4)
    r = orc.to_f32(orc.quant_unpack(codes, meta, 4, 768, 4, "bf16"), "bf16")
    assert ((X - r).view(np.uint32) == e2.view(np.uint32)).all()


@pytest.mark.parametrize("b", [4, 32])
def test_topk_then_quant_composes(orc, b):
    rng = np.random.default_rng(21)
    n_seg, L = 2, 5000
    k = orc.topk_count(L, 1, 10)
    x = orc.from_f32(rng.standard_normal((n_seg, L)).astype(np.float32), "bf16")
    e = (rng.standard_normal((n_seg, L)) * 0.05).astype(np.float32)
    X = orc.to_f32(x, "bf16") + e
    idx, codes, meta, e2 = orc.ef_topk_quant(x, "bf16", e, n_seg, L, k, b)
    idx1, _, _ = orc.ef_topk(x, "bf16", e, n_seg, L, k, wire="f32")
    assert (idx == idx1).all()                                   # same selection as plain TopK
    for s in range(n_seg):
        c2, m2 = orc.quant_pack(X[s][idx[s]], "f32", 1, k, b)   # quantizer on the kept list
        assert (codes[s] == c2[0]).all() and (meta[s] == m2[0]).all()
    y = orc.topk_quant_decompress(idx, codes, meta, n_seg, L, k, b, "bf16")
    r = orc.to_f32(y, "bf16")
    assert ((X - r).view(np.uint32) == e2.view(np.uint32)).all()
    if b == 32:
        kept = np.zeros((n_seg, L), bool)
        for s in range(n_seg):
            kept[s, idx[s]] = True
        assert (y[kept] == orc.from_f32(X, "bf16")[kept]).all() and (y[~kept] == 0).all()
