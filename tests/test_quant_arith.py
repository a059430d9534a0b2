"""Host checks of the binary32 identities the HIP quantizer relies on.

The device quantizer computes the SymQuant scale and codes (APEX4 Sec. 3.2.1)
with a cheaper sequence than the oracle's exact rational arithmetic.  These tests
pin, on the host with IEEE binary32 numpy arithmetic, the facts that make the
two agree bit for bit:

  1. binary16(fl32(amax) * fl32(1/7)) is the binary16 RNE of the exact amax / 7,
     for every positive finite binary16 amax;
  2. (t + 1.5 * 2^23) - 1.5 * 2^23 rounds t to the nearest even integer, and the
     low 4 bits of fl32(t + 1.5 * 2^23) are that integer's two's-complement
     nibble, for t in [-8, 7];
  3. for binary16 x and s, a quotient x / s in [-8.5, 8.5] that is not exactly a
     half-integer is at least 2^-14 away from every half-integer, so an
     approximation within 2^-19 rounds the same way, and one that lands within
     2^-15 of a half-integer is flagged and recomputed exactly.
"""
from fractions import Fraction

import numpy as np

MAGIC = np.float32(12582912.0)


def _exact_rne_f16(fr: Fraction) -> int:
    """Bit pattern of the binary16 nearest to a positive rational (ties to even)."""
    lo = np.float16(float(fr))                       # within one binary16 ulp
    cands = {int(lo.view(np.uint16)) + d for d in (-1, 0, 1)}
    best = None
    for b in sorted(c for c in cands if 0 <= c < 0x7C00):
        v = Fraction(float(np.uint16(b).view(np.float16)))
        key = (abs(v - fr), b & 1)
        if best is None or key < best[0]:
            best = (key, b)
    return best[1]


def test_scale_by_reciprocal_of_seven_is_exact():
    bits = np.arange(1, 0x7C00, dtype=np.uint16)
    a32 = bits.view(np.float16).astype(np.float32)
    got = (a32 * (np.float32(1) / np.float32(7))).astype(np.float16).view(np.uint16)
    # exact reference for every value (rational arithmetic)
    want = np.array([_exact_rne_f16(Fraction(float(a)) / 7) for a in bits.view(np.float16)], np.uint16)
    assert np.array_equal(got, want)


def test_magic_rounding_and_nibble():
    rng = np.random.default_rng(7)
    t = np.concatenate([
        rng.uniform(-8, 7, 2_000_000).astype(np.float32),
        np.arange(-16, 15, dtype=np.float32) / np.float32(2),           # every half-integer in range
        np.nextafter(np.arange(-16, 15, dtype=np.float32) / 2, np.float32(np.inf)),
        np.nextafter(np.arange(-16, 15, dtype=np.float32) / 2, np.float32(-np.inf)),
    ])
    t = np.clip(t, np.float32(-8), np.float32(7))
    r = (t + MAGIC).astype(np.float32)
    q = (r - MAGIC).astype(np.float32)
    assert np.array_equal(q, np.rint(t))                                   # numpy rint: ties to even
    nib = r.view(np.uint32) & 0xF
    assert np.array_equal(nib, np.rint(t).astype(np.int64) & 0xF)


def test_non_tie_quotients_keep_distance_from_half_integers():
    xs = np.arange(0, 0x7C00, dtype=np.uint16)
    x = np.concatenate([xs, xs | 0x8000]).view(np.float16).astype(np.float64)
    rng = np.random.default_rng(11)
    s_bits = np.unique(np.concatenate([
        np.arange(1, 64, dtype=np.uint16),                                 # subnormal scales
        rng.integers(0x0400, 0x7BFF, 300, dtype=np.uint16),                # normal scales
        np.array([0x3C00, 0x4000, 0x4700, 0x2F00, 0x7BFF, 0x0400, 0x03FF], np.uint16),
    ]))
    margin = 2.0 ** -14
    for sb in s_bits:
        s = float(np.uint16(sb).view(np.float16))
        qt = x / s                                                         # binary64, error << 2^-40 here
        inr = np.abs(qt) <= 8.5
        d = np.abs(qt[inr] - (np.floor(qt[inr]) + 0.5))                    # distance to the nearest k + 1/2
        d = np.minimum(d, np.abs(qt[inr] - (np.floor(qt[inr]) - 0.5)))
        tie = d < 2.0 ** -40
        assert np.all(d[~tie] >= margin), f"scale {sb:#06x}"
