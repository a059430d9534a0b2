"""Pins for the oracle's SymQuant (APEX4 Sec. 3.2.1, Eq. SymQuant; Alg. 1).

  * hand-computed worked examples (tests/golden/symquant_worked.json);
  * the binary16 scale S = RNE16(amax / 7) for every positive finite binary16
    amax, against exact rational rounding and against numpy's conversion;
  * the integer code RNE(x / S) for every binary16 x over a spread of scales,
    against numpy's rint of the binary64 quotient (exact for these operands);
  * invariants: max|q| = 7 for a normal scale, |x - q S| <= S/2, sign symmetry,
    power-of-two scale equivariance, the packing layout.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def unpack(q_packed: np.ndarray) -> np.ndarray:
    """[R, K/2] packed bytes -> [R, K] signed codes (low nibble = even k)."""
    lo = (q_packed & 0xF).astype(np.int16)
    hi = (q_packed >> 4).astype(np.int16)
    codes = np.empty(q_packed.shape[:-1] + (q_packed.shape[-1] * 2,), np.int16)
    codes[..., 0::2] = lo
    codes[..., 1::2] = hi
    return np.where(codes >= 8, codes - 16, codes)


def load_cases():
    with open(os.path.join(HERE, "golden", "symquant_worked.json")) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", load_cases(), ids=lambda c: c["name"])
def test_worked_examples(O, case):
    if "x" in case:
        x = np.array(case["x"], np.float64)
        scales = np.array(case["scales"], np.float64)
    else:
        x = np.array(case["x_units_2^-24"], np.float64) * 2.0 ** -24
        scales = np.array(case["scales_units_2^-24"], np.float64) * 2.0 ** -24
    x16 = x.astype(np.float16)
    assert np.array_equal(x16.astype(np.float64), x), "fixture values must be exact binary16"
    q, s = O.quantize(x16[None, :], case["G"])
    assert np.array_equal(s[0].astype(np.float64), scales)
    assert unpack(q)[0].tolist() == case["codes"]
    assert q[0].tobytes().hex() == "".join(case["packed_hex"])


def _positive_finite_f16():
    return np.arange(1, 0x7C00, dtype=np.uint16).view(np.float16)


def test_scale_every_amax_exact_rational(O):
    amax = _positive_finite_f16()
    x = np.stack([amax, np.zeros_like(amax)], axis=1)   # one group of 2 per row
    _, s = O.quantize(x, 2)
    s = s[:, 0]
    # numpy: binary64 quotient then numpy's own binary16 rounding
    assert np.array_equal(s.view(np.uint16), (amax.astype(np.float64) / 7.0).astype(np.float16).view(np.uint16))
    # exact rational nearest binary16, ties to even bit pattern
    grid = np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float64)
    for a, got in zip(amax.astype(np.float64)[::7], s.astype(np.float64)[::7]):
        t = Fraction(float(a)) / 7
        i = int(np.searchsorted(grid, float(t)))
        cands = [j for j in (i - 1, i, i + 1) if 0 <= j < grid.size]
        best = min(cands, key=lambda j: (abs(Fraction(float(grid[j])) - t), j & 1))
        assert got == grid[best]


def test_zero_and_underflow_groups(O):
    u = 2.0 ** -24
    # amax <= 3 * 2^-24: amax/7 < 2^-25 rounds to a zero scale -> zero codes
    x = np.array([[3 * u, -2 * u, u, 0], [0, 0, 0, 0], [4 * u, -4 * u, 2 * u, u]], np.float64).astype(np.float16)
    q, s = O.quantize(x, 4)
    assert s[0, 0] == 0 and s[1, 0] == 0
    assert (unpack(q)[:2] == 0).all()
    # amax = 4 * 2^-24: 4/7 = 0.571 steps -> one step; codes 4,-4,2,1
    assert s[2, 0] == np.float16(u)
    assert unpack(q)[2].tolist() == [4, -4, 2, 1]


def _codes_reference(x: np.ndarray, s: np.ndarray) -> np.ndarray:
    """clip(rint(x/S)) with numpy's binary64 division and rint.

    For binary16 x and S an exact half-integer quotient is representable in
    binary64 and any other quotient lies >= 2^-14 from a half-integer, so this
    is the exact round-half-even of the quotient."""
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.rint(x.astype(np.float64) / s.astype(np.float64))
    r = np.where(s.astype(np.float64) == 0, 0, r)
    return np.clip(r, -8, 7).astype(np.int16)


def test_codes_every_x_for_many_scales(O):
    """Every binary16 x with |x| <= amax, for 160 amax values spread over the range."""
    rng = np.random.default_rng(2024)
    pos = np.arange(1, 0x7C00, dtype=np.uint16)
    picks = np.concatenate([
        rng.choice(pos, 120, replace=False),
        np.arange(1, 40, dtype=np.uint16),               # subnormal amax
        np.array([0x3C00, 0x4700, 0x7BFF], np.uint16),    # 1, 7, 65504
    ])
    allx = np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float64)
    for hb in picks:
        amax = float(np.uint16(hb).view(np.float16))
        mags = allx[allx <= amax]
        vals = np.concatenate([mags, -mags])
        G = 1 << int(np.ceil(np.log2(vals.size + 1)))
        row = np.zeros(G, np.float64)
        row[0] = amax
        row[1:1 + vals.size] = vals
        x = row.astype(np.float16)[None, :]
        q, s = O.quantize(x, G)
        ref = _codes_reference(x[0], np.full(G, s[0, 0]))
        assert np.array_equal(unpack(q)[0], ref), f"amax={amax}"


def test_invariants_random(O):
    rng = np.random.default_rng(5)
    for G in (32, 64, 128, 256, 512):
        x = (rng.standard_normal((64, 2048)) * np.exp2(rng.uniform(-8, 8, size=(64, 1)))).astype(np.float16)
        q, s = O.quantize(x, G)
        c = unpack(q).reshape(64, -1, G)
        s64 = s.astype(np.float64)
        normal = s64 >= 2.0 ** -14
        assert normal.all()
        assert (np.abs(c).max(axis=2) == 7).all()            # the max element maps to +-7
        xr = x.astype(np.float64).reshape(64, -1, G)
        assert (np.abs(xr - c * s64[..., None]) <= s64[..., None] / 2).all()
        assert (c >= -7).all()                                # -8 needs a subnormal scale
        # sign symmetry and power-of-two equivariance
        qn, sn = O.quantize(-x, G)
        assert np.array_equal(unpack(qn), -unpack(q)) and np.array_equal(sn, s)
        q2, s2 = O.quantize((x.astype(np.float32) * 4).astype(np.float16), G)
        assert np.array_equal(unpack(q2), unpack(q)) and np.array_equal(s2.astype(np.float64), 4 * s64)


def test_per_channel_group_is_whole_row(O):
    rng = np.random.default_rng(9)
    x = rng.standard_normal((8, 512)).astype(np.float16)
    q, s = O.quantize(x, 512)
    assert s.shape == (8, 1)
    amax = np.abs(x.astype(np.float64)).max(axis=1)
    assert np.array_equal(s[:, 0].view(np.uint16), (amax / 7.0).astype(np.float16).view(np.uint16))
    assert np.array_equal(unpack(q), _codes_reference(x, np.repeat(s, 512, axis=1)))


def test_packing_layout(O):
    # codes 1, -1 -> byte 0xF1 (low nibble holds the even k)
    x = np.array([[7.0, -7.0, 1.0, -1.0]], np.float16)
    q, s = O.quantize(x, 4)
    assert s[0, 0] == 1.0 and q[0].tobytes() == bytes([0x97, 0xF1])
