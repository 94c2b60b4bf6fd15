"""Pins for the oracle's TopK at given indices (Sec. 3.2: in the GPT-2 runs the
gradients are compressed at the indices the activations' TopK kept, instead of
a selection of their own), alone and inside error feedback (Sec. 2.4).

Checked against: the oracle's own TopK (gathering a tensor at the indices of
its TopK must give back exactly that TopK's values), numpy's masking and
IEEE binary16 conversion for the dense reconstruction and the residual,
exact telescoping of the sent values plus the final residual over several
steps (binary32 wire, values exactly representable), and the edge cases
(k = 0, an index outside the segment)."""
import numpy as np
import pytest


def _mask(idx, n_seg, L):
    m = np.zeros((n_seg, L), bool)
    for s in range(n_seg):
        m[s, idx[s]] = True
    return m


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("L,k", [(1, 1), (37, 5), (1000, 100), (5000, 1500)])
def test_gather_at_own_topk_is_topk(orc, dt, L, k):
    rng = np.random.default_rng(L + k)
    x = rng.standard_normal((3, L)).astype(np.float32)
    x[:, ::7] = 0.0
    xr = orc.from_f32(x, dt) if dt != "f32" else x
    idx, val = orc.topk_compress(xr, dt, 3, L, k)
    g = orc.topk_gather(xr, dt, idx, 3, L, k)
    assert g.dtype == val.dtype and np.array_equal(g.view(np.uint8), val.view(np.uint8))


def test_gather_reconstruction_is_masking(orc):
    rng = np.random.default_rng(3)
    n_seg, L, k = 4, 777, 80
    g = rng.standard_normal((n_seg, L)).astype(np.float32)
    # indices from an unrelated tensor: the forward activations
    idx, _ = orc.topk_compress(rng.standard_normal((n_seg, L)).astype(np.float32), "f32", n_seg, L, k)
    g16 = g.astype(np.float16)
    val = orc.topk_gather(g16.view(np.uint16), "f16", idx, n_seg, L, k)
    y = orc.topk_decompress(idx, val, "f16", n_seg, L, k, out_dt="f32")
    expect = np.where(_mask(idx, n_seg, L), g16.astype(np.float32), np.float32(0.0))
    assert np.array_equal(y.view(np.uint32), expect.view(np.uint32))


def test_gather_ef_residual_f16(orc):
    rng = np.random.default_rng(4)
    n_seg, L, k = 3, 640, 64
    x = rng.standard_normal((n_seg, L)).astype(np.float32)
    e = (1e-3 * rng.standard_normal((n_seg, L))).astype(np.float32)
    idx, _ = orc.topk_compress(rng.standard_normal((n_seg, L)).astype(np.float32), "f32", n_seg, L, k)
    x16 = x.astype(np.float16)
    val, e2 = orc.topk_gather(x16.view(np.uint16), "f16", idx, n_seg, L, k, e=e)
    X = x16.astype(np.float32) + e
    sent = X.astype(np.float16).astype(np.float32)
    m = _mask(idx, n_seg, L)
    expect = np.where(m, X - sent, X - np.float32(0.0)).astype(np.float32)
    assert np.array_equal(e2.view(np.uint32), expect.view(np.uint32))
    assert np.array_equal(val.view(np.float16).astype(np.float32)[0],
                          X[0, idx[0]].astype(np.float16).astype(np.float32))


def test_gather_ef_telescopes(orc):
    # binary32 wire and small integers: every sum below is exact, so
    # sum of received tensors + final residual == sum of inputs, bitwise
    rng = np.random.default_rng(5)
    n_seg, L, k, steps = 2, 300, 40, 5
    e = np.zeros((n_seg, L), np.float32)
    got = np.zeros((n_seg, L), np.float64)
    total = np.zeros((n_seg, L), np.float64)
    for t in range(steps):
        x = rng.integers(-50, 50, (n_seg, L)).astype(np.float32)
        idx, _ = orc.topk_compress(rng.standard_normal((n_seg, L)).astype(np.float32), "f32", n_seg, L, k)
        val, e = orc.topk_gather(x, "f32", idx, n_seg, L, k, e=e)
        y = orc.topk_decompress(idx, val, "f32", n_seg, L, k)
        got += y
        total += x
        # at the sent indices nothing is left behind
        assert np.all(e[_mask(idx, n_seg, L)] == 0.0)
    assert np.array_equal(got + e, total)


def test_gather_edges(orc):
    x = np.arange(10, dtype=np.float32)
    e = np.ones((1, 10), np.float32)
    val, e2 = orc.topk_gather(x, "f32", np.zeros((1, 0), np.uint32), 1, 10, 0, e=e)
    assert val.shape == (1, 0) and np.array_equal(e2, (x + 1.0).reshape(1, 10))
    with pytest.raises(ValueError):
        orc.topk_gather(x, "f32", np.array([[3, 10]], np.uint32), 1, 10, 2)
