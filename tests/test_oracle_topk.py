"""Pins for the oracle's TopK (Sec. 2.3: keep the K% entries of largest absolute
value, zero the rest; indices are sent with the values, Sec. 4.1).

Checked against: the hand-worked example in tests/golden/topk_w1.txt, a
brute-force search over all index subsets for tiny inputs (the subset that
satisfies the defining dominance + lower-index-on-ties property is unique),
invariants at larger sizes on tie-heavy data, the k = 0 / k = L special cases,
and exact rational ceilings for the K% -> k count.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest

from conftest import read_golden


def test_worked_example_w1(orc):
    g = read_golden("topk_w1.txt")
    v = np.array([float(t) for t in g["v"]], np.float32)
    assert np.signbit(v[4]) and not np.signbit(v[3])
    for k in (3, 5, 6, 7):
        idx = orc.topk_indices(v, k)
        assert idx.tolist() == [int(t) for t in g[f"k{k}_idx"]]
    idx, val = orc.topk_compress(v, "f32", 1, v.size, 3)
    assert val[0].tolist() == [float(t) for t in g["k3_val"]]
    idx, val = orc.topk_compress(v, "f32", 1, v.size, 6)
    assert val[0].tolist() == [float(t) for t in g["k6_val"]]
    # the kept zero is +0 (index 3), not the -0 of index 4
    assert not np.signbit(val[0][3])


def _valid_sets(mag, k):
    """all k-subsets S with: i in S, j not in S => |v_i| > |v_j| or (|v_i| == |v_j| and i < j)"""
    n = len(mag)
    out = []
    for S in itertools.combinations(range(n), k):
        s = set(S)
        ok = all(mag[i] > mag[j] or (mag[i] == mag[j] and i < j)
                 for i in S for j in range(n) if j not in s)
        if ok:
            out.append(list(S))
    return out


ALPHABET = np.array([0.0, -0.0, 1.0, -1.0, 2.0, -2.0, 3.0], np.float32)


def test_bruteforce_exhaustive_small(orc):
    # every vector of length <= 5 over {+0,-0,+-1,+-2,3}, every k
    for n in range(0, 6):
        for combo in itertools.product(range(len(ALPHABET)), repeat=n):
            v = ALPHABET[list(combo)]
            mag = [abs(float(t)) for t in v]
            for k in range(0, n + 1):
                sets = _valid_sets(mag, k)
                assert len(sets) == 1
                assert orc.topk_indices(v, k).tolist() == sets[0]


def test_bruteforce_random_up_to_9(orc):
    rng = np.random.default_rng(7)
    for _ in range(400):
        n = int(rng.integers(5, 10))
        v = ALPHABET[rng.integers(0, len(ALPHABET), size=n)]
        mag = [abs(float(t)) for t in v]
        k = int(rng.integers(0, n + 1))
        sets = _valid_sets(mag, k)
        assert len(sets) == 1
        assert orc.topk_indices(v, k).tolist() == sets[0]


def _check_invariants(v, k, idx):
    mag = np.abs(v.astype(np.float64))
    assert idx.size == k
    assert (np.diff(idx.astype(np.int64)) > 0).all()          # ascending, distinct
    if k == 0 or k == v.size:
        return
    kept = np.zeros(v.size, bool)
    kept[idx] = True
    T = mag[kept].min()
    assert T >= mag[~kept].max()                              # dominance
    # among entries equal to the threshold, exactly the lowest indices are kept
    ties = np.flatnonzero(mag == T)
    r = k - int((mag > T).sum())
    assert kept[ties[:r]].all() and not kept[ties[r:]].any()


@pytest.mark.parametrize("n,seed", [(1000, 0), (4096, 1), (4097, 2), (12345, 3)])
def test_invariants_tie_heavy(orc, n, seed):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal(n).astype(np.float32)
    # bfloat16-rounded magnitudes and 50% exact zeros (both signs): many ties
    z = z.astype(np.float32).view(np.uint32) & np.uint32(0xFFFF0000)
    z = z.view(np.float32)
    z[rng.random(n) < 0.5] = 0.0
    z[rng.random(n) < 0.1] = -0.0
    for k in sorted({0, 1, n // 10, n // 3, n // 2, n // 2 + 7, n - 1, n}):
        _check_invariants(z, k, orc.topk_indices(z, k))


def test_k_zero_and_full(orc):
    rng = np.random.default_rng(11)
    x = rng.standard_normal((3, 100)).astype(np.float32)
    x[0, 5] = -0.0
    # k = 0: empty payload, dense output all +0
    idx, val = orc.topk_compress(x, "f32", 3, 100, 0)
    y = orc.topk_decompress(idx, val, "f32", 3, 100, 0)
    assert (y.view(np.uint32) == 0).all()
    # k = L: identity, bit for bit (the -0 survives)
    idx, val = orc.topk_compress(x, "f32", 3, 100, 100)
    y = orc.topk_decompress(idx, val, "f32", 3, 100, 100)
    assert (y.view(np.uint32) == x.view(np.uint32)).all()


@pytest.mark.parametrize("dt", ["bf16", "f16"])
def test_half_inputs_wire_is_input_dtype(orc, dt):
    rng = np.random.default_rng(5)
    x32 = rng.standard_normal((4, 333)).astype(np.float32)
    x = orc.from_f32(x32, dt)
    k = orc.topk_count(333, 1, 10)
    idx, val = orc.topk_compress(x, dt, 4, 333, k)
    # the kept values are the inputs themselves (an exact upcast and back)
    for s in range(4):
        assert (val[s] == x[s][idx[s]]).all()
    y = orc.topk_decompress(idx, val, dt, 4, 333, k)
    keep = np.zeros((4, 333), bool)
    for s in range(4):
        keep[s, idx[s]] = True
    assert (y[keep] == x[keep]).all() and (y[~keep] == 0).all()


def test_topk_count_is_exact_ceiling(orc):
    rng = np.random.default_rng(3)
    cases = [(100, 7, 100), (100, 3, 10), (16384, 1, 10), (32768, 3, 10), (768, 1, 10),
             (393216, 3, 10), (2 ** 27, 1, 10), (0, 1, 10), (5, 0, 1), (5, 1, 1)]
    cases += [(int(rng.integers(0, 10 ** 9)), int(rng.integers(0, 1000)), int(rng.integers(1, 1000)))
              for _ in range(2000)]
    for L, num, den in cases:
        want = -((-Fraction(L * num, den).numerator) // Fraction(L * num, den).denominator)
        assert orc.topk_count(L, num, den) == want
    # the K% -> k figures of the boundary workloads
    assert orc.topk_count(16384, 1, 10) == 1639
    assert orc.topk_count(32768, 3, 10) == 9831
    assert orc.topk_count(768, 1, 10) == 77
    assert orc.topk_count(393216, 3, 10) == 117965
    assert orc.topk_count(2 ** 27, 1, 10) == 13421773
    assert orc.topk_count(100, 7, 100) == 7
    assert orc.topk_count(100, 3, 10) == 30
