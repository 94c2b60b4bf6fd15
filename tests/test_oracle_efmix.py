"""Pins for the oracle's EF-mixed compressor (Sec. 2.4: half of the TopK budget
goes to the largest entries of the input, half to the largest entries of the
error buffer; both are sent and added).

Checked against: a worked example computed by hand (two steps, with an index
picked by both halves and a tie broken towards the lower index), numpy
selections of the largest magnitudes, exact conservation x + e = received + e'
on integer data (every sum exact), the bfloat16 rounding remainder of a sent
buffer entry written out by hand, an index held by both lists whose received
sum rounds in the wire dtype (worked by hand, and conservation on
non-integer data where every binary32 operation is exact but the wire's
roundings are not), and the edge cases (k = 0, 1 and L, the first step from an
empty buffer, an index outside the segment)."""
import numpy as np
import pytest


def _topk_np(v, k):
    """indices (ascending) of the k largest |v|, ties to the lower index"""
    order = np.lexsort((np.arange(v.size), -np.abs(v.astype(np.float64))))
    return np.sort(order[:k]).astype(np.uint32)


def test_counts(orc):
    assert orc.efmix_counts(0) == (0, 0)
    assert orc.efmix_counts(1) == (1, 0)
    assert orc.efmix_counts(4) == (2, 2)
    assert orc.efmix_counts(3277) == (1639, 1638)


def test_worked_example_two_steps(orc):
    # step 1: k = 4 on 8 entries -> 2 from x, 2 from e, disjoint
    x1 = np.array([[3, -1, 0.5, -7, 2, 0, 4, -2]], np.float32)
    e0 = np.array([[0, 5, 0, -1, 0, 0.25, 0, 3]], np.float32)
    ix, vx, ie, ve, e1 = orc.efmix_send(x1, "f32", e0, 1, 8, 4)
    assert ix.tolist() == [[3, 6]] and vx.tolist() == [[-7, 4]]
    assert ie.tolist() == [[1, 7]] and ve.tolist() == [[5, 3]]
    y = orc.efmix_recv(ix, vx, ie, ve, "f32", 1, 8, 4)
    assert y.tolist() == [[0, 5, 0, -7, 0, 0, 4, 3]]
    assert e1.tolist() == [[3, -1, 0.5, -1, 2, 0.25, 0, -2]]
    # step 2: both halves pick index 0; |e| ties at 2 (indices 4 and 7): 4 wins
    x2 = np.array([[1, 0, 0, 0, 0, 0, 0, 9]], np.float32)
    ix, vx, ie, ve, e2 = orc.efmix_send(x2, "f32", e1, 1, 8, 4)
    assert ix.tolist() == [[0, 7]] and vx.tolist() == [[1, 9]]
    assert ie.tolist() == [[0, 4]] and ve.tolist() == [[3, 2]]
    y = orc.efmix_recv(ix, vx, ie, ve, "f32", 1, 8, 4)
    assert y.tolist() == [[4, 0, 0, 0, 2, 0, 0, 9]]
    assert e2.tolist() == [[0, -1, 0.5, -1, 0, 0.25, 0, -2]]


@pytest.mark.parametrize("dt", ["f32", "f16"])
@pytest.mark.parametrize("L,num", [(64, 1), (1000, 3), (4097, 1)])
def test_integer_conservation_and_selection(orc, dt, L, num):
    # integers below 2^10: every value, wire value and sum is exact, so
    # x + e == received + e' holds bit for bit at every step
    rng = np.random.default_rng(L * 7 + num)
    n_seg, k = 3, orc.topk_count(L, num, 10)
    kx, ke = orc.efmix_counts(k)
    e = np.zeros((n_seg, L), np.float32)
    for step in range(4):
        x = rng.integers(-60, 61, (n_seg, L)).astype(np.float32)
        xr = x.astype(np.float16).view(np.uint16) if dt == "f16" else x
        ix, vx, ie, ve, e_next = orc.efmix_send(xr, dt, e, n_seg, L, k)
        y = orc.efmix_recv(ix, vx, ie, ve, dt, n_seg, L, k, out_dt="f32")
        for s in range(n_seg):
            assert np.array_equal(ix[s], _topk_np(x[s], kx)), f"S_x step {step}"
            assert np.array_equal(ie[s], _topk_np(e[s], ke)), f"S_e step {step}"
        assert np.array_equal(x + e, y + e_next), f"conservation step {step}"
        assert ((y != 0).sum(axis=1) <= k).all()
        e = e_next


def test_bf16_wire_remainder_stays_in_buffer(orc):
    # e = 1 + 2^-10 rounds to 1.0 in bfloat16 (8 significant bits): the sent
    # value is 1.0 (0x3F80) and 2^-10 stays in the buffer
    L, k = 4, 2
    xr = np.zeros((1, L), np.uint16)   # x = +0 in bfloat16
    e = np.array([[0.0, 1.0 + 2.0 ** -10, 0.0, 0.0]], np.float32)
    ix, vx, ie, ve, e1 = orc.efmix_send(xr, "bf16", e, 1, L, k)
    assert ie.tolist() == [[1]] and ve.tolist() == [[0x3F80]]
    assert ix.tolist() == [[0]]
    assert e1.tolist() == [[0.0, 2.0 ** -10, 0.0, 0.0]]
    y = orc.efmix_recv(ix, vx, ie, ve, "bf16", 1, L, k, out_dt="f32")
    assert y.tolist() == [[0.0, 1.0, 0.0, 0.0]]


def test_shared_index_keeps_what_the_receivers_rounding_drops(orc):
    # index 0 is the largest entry of both x and e.  The receiver holds
    # bf16(1 + 2^-8): 1 + 2^-8 lies halfway between 1 and 1 + 2^-7 and rounds
    # to the even neighbour 1.0, so the buffer must keep 2^-8 there
    L, k = 4, 2
    x = np.array([[1.0, 0.25, -0.5, 0.125]], np.float32)
    xr = (x.view(np.uint32) >> 16).astype(np.uint16)      # exact in bfloat16
    e = np.array([[2.0 ** -8, 0.0, 0.0, 0.0]], np.float32)
    ix, vx, ie, ve, e1 = orc.efmix_send(xr, "bf16", e, 1, L, k)
    assert ix.tolist() == [[0]] and ie.tolist() == [[0]]
    assert vx.tolist() == [[0x3F80]] and ve.tolist() == [[0x3B80]]   # 1.0 and 2^-8
    y = orc.efmix_recv(ix, vx, ie, ve, "bf16", 1, L, k, out_dt="bf16")
    assert y.tolist() == [[0x3F80, 0, 0, 0]]
    assert e1.tolist() == [[2.0 ** -8, 0.25, -0.5, 0.125]]


def orc_round(v, dt):
    """round binary32 to the wire dtype (RNE) with numpy alone, back to binary32"""
    v = np.asarray(v, np.float32)
    if dt == "f16":
        return v.astype(np.float16).astype(np.float32)
    b = v.view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16 << 16
    return b.astype(np.uint32).view(np.float32)


def _wire_bits(v, dt):
    """binary32 values exact in dt -> the dt's raw pattern"""
    if dt == "f16":
        return v.astype(np.float16).view(np.uint16)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def _to_f32(r, dt):
    if dt == "f16":
        return r.view(np.float16).astype(np.float32)
    return (r.astype(np.uint32) << 16).view(np.float32)


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_conservation_with_shared_indices_off_the_wire_grid(orc, dt):
    # values are multiples of 2^-6 below 2^9 in magnitude: every binary32
    # sum and difference below is exact, while the wire dtype keeps only 8
    # (bf16) or 11 (f16) significant bits.  The buffer is largest where x is,
    # so the two lists share indices, and their sums fall off the wire's grid.
    # With the receiver in the wire dtype, x + e == received + e' must hold
    # bit for bit; dropping c_i (the receiver's rounding at shared indices)
    # breaks it.
    rng = np.random.default_rng(77 if dt == "bf16" else 78)
    n_seg, L, k = 2, 4000, 800
    e = (rng.integers(-2 ** 12, 2 ** 12, (n_seg, L)) / 64.0).astype(np.float32)
    shared_off_grid = 0
    for step in range(4):
        x = orc_round((rng.integers(-2 ** 10, 2 ** 10, (n_seg, L)) / 64.0).astype(np.float32), dt)
        hot = np.argsort(-np.abs(e), axis=1)[:, : k // 3]     # x large where e is
        np.put_along_axis(x, hot, orc_round(np.take_along_axis(e, hot, 1) * 0.75 + 3.0, dt), 1)
        ix, vx, ie, ve, e_next = orc.efmix_send(_wire_bits(x, dt), dt, e, n_seg, L, k)
        y = orc.efmix_recv(ix, vx, ie, ve, dt, n_seg, L, k, out_dt=dt)
        yf = _to_f32(y, dt)
        assert np.array_equal((x + e).view(np.uint32), (yf + e_next).view(np.uint32)), f"step {step}"
        for s in range(n_seg):
            both = np.intersect1d(ix[s], ie[s])
            u = x[s, both] + orc_round(e[s, both], dt)
            shared_off_grid += int((orc_round(u, dt) != u).sum())
        e = e_next
    assert shared_off_grid > 50


def test_first_step_from_empty_buffer(orc):
    # e = 0: the e half picks the k_e lowest indices (all |e| tie) and sends
    # +0; the buffer becomes x off the x half's indices
    rng = np.random.default_rng(5)
    n_seg, L, k = 2, 300, 60
    kx, ke = orc.efmix_counts(k)
    x = rng.standard_normal((n_seg, L)).astype(np.float32)
    ix, vx, ie, ve, e1 = orc.efmix_send(x, "f32", np.zeros((n_seg, L), np.float32), n_seg, L, k)
    for s in range(n_seg):
        assert np.array_equal(ie[s], np.arange(ke, dtype=np.uint32))
        assert (ve[s] == 0).all()
        m = np.zeros(L, bool)
        m[ix[s]] = True
        assert np.array_equal(e1[s], np.where(m, 0.0, x[s]).astype(np.float32))
        assert np.array_equal(vx[s], x[s, ix[s]])


@pytest.mark.parametrize("k", [0, 1, 7])
def test_small_budgets(orc, k):
    rng = np.random.default_rng(k)
    L = 7
    x = rng.standard_normal((2, L)).astype(np.float32)
    e = rng.standard_normal((2, L)).astype(np.float32)
    kx, ke = orc.efmix_counts(k)
    ix, vx, ie, ve, e1 = orc.efmix_send(x, "f32", e, 2, L, k)
    assert ix.shape == (2, kx) and ie.shape == (2, ke)
    y = orc.efmix_recv(ix, vx, ie, ve, "f32", 2, L, k)
    if k == 0:
        assert (y == 0).all() and np.array_equal(e1, x + e)
    for s in range(2):
        assert np.array_equal(ix[s], _topk_np(x[s], kx))
        assert np.array_equal(ie[s], _topk_np(e[s], ke))
    # off both index sets the buffer holds x + e; on them what was not sent
    for s in range(2):
        only = np.setdiff1d(np.arange(L), np.union1d(ix[s], ie[s]))
        assert np.array_equal(e1[s, only], x[s, only] + e[s, only])
        both = np.intersect1d(ix[s], ie[s])
        assert (e1[s, both] == 0).all()


def test_bad_index_rejected(orc):
    ix = np.array([[9]], np.uint32)
    vx = np.array([[1.0]], np.float32)
    ie = np.zeros((1, 0), np.uint32)
    ve = np.zeros((1, 0), np.float32)
    with pytest.raises(ValueError):
        orc.efmix_recv(ix, vx, ie, ve, "f32", 1, 8, 1)
