"""Pins for the oracle's binary16 converters (IEEE 754-2008 binary16).

The oracle writes both conversions out from the format definition; these tests
hold them against numpy's conversions (a library routine) and against exact
rational rounding, exhaustively where the domain is small.
"""
from fractions import Fraction

import numpy as np


def all_f16_patterns():
    return np.arange(65536, dtype=np.uint32).astype(np.uint16)


def test_f16_to_f64_exhaustive(O):
    h = all_f16_patterns()
    got = O.f16_to_f64(h)
    ref = h.view(np.float16).astype(np.float64)
    same = (got == ref) | (np.isnan(got) & np.isnan(ref))
    assert same.all()
    # signed zeros keep their sign
    assert np.signbit(got[0x8000]) and not np.signbit(got[0])


def _finite_positive_f16():
    h = np.arange(0, 0x7C00, dtype=np.uint16)
    return h.view(np.float16).astype(np.float64)


def test_f64_to_f16_roundtrip_every_value(O):
    h = all_f16_patterns()
    v = h.view(np.float16).astype(np.float64)
    finite = np.isfinite(v)
    back = O.f64_to_f16(v[finite]).view(np.uint16)
    assert np.array_equal(back, h[finite])


def test_f64_to_f16_midpoints_tie_to_even(O):
    v = _finite_positive_f16()
    mids = (v[:-1] + v[1:]) / 2.0                   # exact in binary64
    lo_bits = np.arange(0, 0x7C00 - 1, dtype=np.uint16)
    # the even bit pattern of the two neighbours wins a tie
    expect = np.where(lo_bits % 2 == 0, lo_bits, lo_bits + 1).astype(np.uint16)
    for sign in (1.0, -1.0):
        got = O.f64_to_f16(sign * mids).view(np.uint16) & 0x7FFF
        assert np.array_equal(got, expect)
    # one binary64 ulp either side of a midpoint is no longer a tie
    up = np.nextafter(mids, np.inf)
    dn = np.nextafter(mids, -np.inf)
    assert np.array_equal(O.f64_to_f16(up).view(np.uint16), lo_bits + 1)
    assert np.array_equal(O.f64_to_f16(dn).view(np.uint16), lo_bits)
    # numpy agrees on all of them
    for arr in (mids, -mids, up, dn):
        assert np.array_equal(O.f64_to_f16(arr).view(np.uint16), arr.astype(np.float16).view(np.uint16))


def test_f64_to_f16_random_vs_numpy(O):
    rng = np.random.default_rng(1234)
    mag = np.exp2(rng.uniform(-30, 17.5, size=2_000_000))
    x = mag * rng.choice([-1.0, 1.0], size=mag.size)
    got = O.f64_to_f16(x).view(np.uint16)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, ref)


def test_f64_to_f16_exact_rational_sample(O):
    """Nearest binary16 by exact rational comparison, for a random sample."""
    rng = np.random.default_rng(7)
    grid = _finite_positive_f16()
    xs = np.exp2(rng.uniform(-26, 15.9, size=3000))
    got = O.f64_to_f16(xs).astype(np.float64)
    for x, g in zip(xs, got):
        i = np.searchsorted(grid, x)
        cands = [grid[j] for j in (i - 1, i) if 0 <= j < grid.size]
        fx = Fraction(float(x))
        best = min(cands, key=lambda c: (abs(Fraction(float(c)) - fx),
                                         int(np.float16(c).view(np.uint16)) & 1))
        assert g == best


def test_f64_to_f16_specials(O):
    cases = [
        (0.0, 0x0000), (-0.0, 0x8000), (np.inf, 0x7C00), (-np.inf, 0xFC00),
        (65504.0, 0x7BFF), (65519.99, 0x7BFF), (65520.0, 0x7C00), (1e6, 0x7C00),
        (2.0 ** -24, 0x0001), (2.0 ** -25, 0x0000), (1.5 * 2.0 ** -25, 0x0001),
        (2.0 ** -14, 0x0400), (1.0, 0x3C00), (-2.0, 0xC000),
    ]
    for x, bits in cases:
        assert int(O.f64_to_f16(np.array([x])).view(np.uint16)[0]) == bits, x
    assert np.isnan(O.f64_to_f16(np.array([np.nan])).astype(np.float64)[0])
