"""Pins for the oracle's AQ-SGD with TopK (Sec. 2.5: one buffer per training
example; the change of the activation against it is compressed with TopK and
sent; both sides fold the message into their copy of the buffer).

Checked against: the hand-worked example tests/golden/aqsgd_w7.txt; the
sender's and receiver's buffers staying bit-identical; rows outside the
micro-batch untouched; a zero buffer reducing AQ-SGD to plain TopK; K = 100%
with a zero buffer being the identity; the sent indices being the TopK of the
delta computed independently in numpy.
"""
import numpy as np
import pytest

from conftest import read_golden


def test_worked_example_w7(orc):
    g = read_golden("aqsgd_w7.txt")
    f = lambda k: np.array([float(t) for t in g[k]], np.float32)
    m = orc.from_f32(np.stack([f("m0"), f("m1")]), "f16")
    m_r = m.copy()
    a = orc.from_f32(f("a")[None], "f16")
    k = int(g["k"][0])
    idx, val = orc.aqsgd_send(a, m, "f16", np.array([1]), k)
    assert idx[0].tolist() == [int(t) for t in g["idx"]]
    assert orc.to_f32(val, "f16")[0].tolist() == f("val").tolist()
    a_hat = orc.aqsgd_recv(idx, val, m_r, "f16", np.array([1]), k)
    assert orc.to_f32(m, "f16")[1].tolist() == f("m1_after").tolist()
    assert orc.to_f32(m, "f16")[0].tolist() == f("m0").tolist()
    assert (a_hat[0] == m[1]).all() and (m_r == m).all()


@pytest.mark.parametrize("dt", ["f16", "f32", "bf16"])
def test_buffers_stay_identical(orc, dt):
    rng = np.random.default_rng(5)
    n_samples, L, B = 32, 777, 4
    k = orc.topk_count(L, 3, 10)
    z = rng.standard_normal((n_samples, L)).astype(np.float32)
    m = z if dt == "f32" else orc.from_f32(z, dt)
    m = np.ascontiguousarray(m)
    m_r = m.copy()
    for step in range(6):
        ids = rng.permutation(n_samples)[:B]
        before = m.copy()
        a32 = orc.to_f32(m[ids], dt) + (rng.standard_normal((B, L)) * 0.1).astype(np.float32)
        a = a32 if dt == "f32" else orc.from_f32(a32, dt)
        d = orc.to_f32(a, dt) - orc.to_f32(m[ids], dt)          # the delta, computed here
        idx, val = orc.aqsgd_send(a, m, dt, ids, k)
        a_hat = orc.aqsgd_recv(idx, val, m_r, dt, ids, k)
        assert (m == m_r).all()
        others = np.setdiff1d(np.arange(n_samples), ids)
        assert (m[others] == before[others]).all()
        for b in range(B):
            mag = np.abs(d[b].astype(np.float64))
            kept = np.zeros(L, bool)
            kept[idx[b]] = True
            assert idx[b].size == k and mag[kept].min() >= mag[~kept].max()
            assert (a_hat[b] == m[ids[b]]).all()
            assert (m[ids[b]][~kept] == before[ids[b]][~kept]).all()


def test_zero_buffer_reduces_to_topk(orc):
    rng = np.random.default_rng(6)
    n_samples, L, B = 10, 1000, 3
    k = orc.topk_count(L, 3, 10)
    m = np.zeros((n_samples, L), np.uint16)              # +0 in binary16
    m_r = m.copy()
    a = orc.from_f32(rng.standard_normal((B, L)).astype(np.float32), "f16")
    ids = np.array([7, 0, 4])
    idx, val = orc.aqsgd_send(a, m, "f16", ids, k)
    a_hat = orc.aqsgd_recv(idx, val, m_r, "f16", ids, k)
    idx2, val2 = orc.topk_compress(a, "f16", B, L, k)
    y = orc.topk_decompress(idx2, val2, "f16", B, L, k)
    assert (idx == idx2).all() and (val == val2).all() and (a_hat == y).all()
    # K = 100% from a zero buffer hands on the activation itself
    m = np.zeros((n_samples, L), np.uint16)
    m_r = m.copy()
    idx, val = orc.aqsgd_send(a, m, "f16", ids, L)
    a_hat = orc.aqsgd_recv(idx, val, m_r, "f16", ids, L)
    assert (a_hat == a).all()


def test_rejects_out_of_range_ids(orc):
    m = np.zeros((4, 8), np.uint16)
    a = np.zeros((1, 8), np.uint16)
    with pytest.raises(ValueError):
        orc.aqsgd_send(a, m, "f16", np.array([4]), 2)


def test_ef21_reaches_a_fixed_input(orc):
    # EF21 (Sec. 2.4): g <- g + C(x - g) is AQ-SGD with one buffer row per
    # segment.  With binary32 values and x held fixed, each step sends the k
    # largest remaining differences exactly, so the difference shrinks and g
    # equals x after ceil(L / k) steps, on both sides
    rng = np.random.default_rng(11)
    B, L, k = 3, 500, 60
    x = rng.standard_normal((B, L)).astype(np.float32)
    g = np.zeros((B, L), np.float32)
    g_r = g.copy()
    ids = np.arange(B)
    prev = np.abs(x - g).sum()
    for t in range(-(-L // k)):
        before = g.copy()
        idx, val = orc.aqsgd_send(x, g, "f32", ids, k)
        orc.aqsgd_recv(idx, val, g_r, "f32", ids, k)
        assert (g == g_r).all()
        for b in range(B):
            # the message is the difference at the sent indices
            assert (val[b] == (x[b] - before[b])[idx[b]]).all()
        diff = np.abs(x - g).sum()
        assert diff < prev or diff == 0.0
        prev = diff
    assert (g == x).all()
