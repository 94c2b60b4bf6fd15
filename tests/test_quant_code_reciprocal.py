"""The quantization sender's encode takes (v - lo) * RN(1 / range) in place
of the correctly rounded quotient, and divides only where the scaled value
lies within 2^-10 of a half-integer (Sec. 2.2's codes must not change).  This
checks that argument in IEEE binary32 arithmetic (numpy float32, one rounding
per operation, as the kernel's code is compiled without contraction) on many
groups, with values spread over the range and values piled up at the
rounding ties."""
import numpy as np
import pytest


def code_direct(v, lo, rng, LV):
    u = (v - lo) / rng
    return np.minimum(np.rint(u * np.float32(LV)), np.float32(LV)).astype(np.uint32)


def code_fast(v, lo, rng, LV):
    n = v - lo
    rcp = np.float32(1.0) / rng
    t = (n * rcp) * np.float32(LV)
    r = np.rint(t)
    ok = np.abs(t - r) < np.float32(0.5 - 2.0 ** -10)
    out = code_direct(v, lo, rng, LV)
    fast = np.minimum(r, np.float32(LV)).astype(np.uint32)
    return np.where(ok, fast, out), ok, fast


@pytest.mark.parametrize("b", [1, 2, 3, 4, 5, 6, 7, 8])
def test_reciprocal_form_gives_the_same_codes(b):
    LV = (1 << b) - 1
    rng_ = np.random.default_rng(100 + b)
    checked = 0
    unguarded_wrong = 0
    for g in range(200):
        lo = np.float32(rng_.normal() * 10.0 ** rng_.integers(-6, 6))
        rng = np.float32(abs(rng_.normal()) * 10.0 ** rng_.integers(-30, 30)) + np.float32(1e-30)
        hi = np.float32(lo + rng)
        rng = np.float32(hi - lo)
        if not (rng > 0) or not (2.0 ** -125 <= rng <= 2.0 ** 125):
            continue
        # values over [lo, hi] and values at the half-integer ties, +- a few ulps
        spread = (lo + rng_.random(4000).astype(np.float32) * rng).astype(np.float32)
        k = rng_.integers(0, LV, 4000)
        ties = (lo + ((k + 0.5) * (np.float64(rng) / LV))).astype(np.float32)
        shift = rng_.integers(-4, 5, 4000)
        for _ in range(4):
            up, dn = shift > 0, shift < 0
            ties[up] = np.nextafter(ties[up], np.float32(np.inf))
            ties[dn] = np.nextafter(ties[dn], np.float32(-np.inf))
            shift = shift - np.sign(shift)
        v = np.concatenate([spread, ties, [lo, hi]]).astype(np.float32)
        v = np.clip(v, lo, hi)
        got, ok, fast = code_fast(v, lo, rng, LV)
        direct = code_direct(v, lo, rng, LV)
        assert np.array_equal(got, direct), (b, g, lo, rng)
        checked += int(ok.sum())
        unguarded_wrong += int((fast != direct).sum())
    assert checked > 100000   # the fast form decided most of them
    # and without the guard it would have been wrong at some ties
    assert unguarded_wrong > 0
