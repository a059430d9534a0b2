"""Pins of the oracle's FP6 e3m2 container (oracle/fp6.py), CPU only.

The decoder is checked against values the OCP Microscaling specification fixes
for e3m2 (largest normal 28, smallest normal 2^-2, smallest subnormal 2^-4,
1.0 = exponent field 3); the encoder against the decoder over every code; the
row layout against big-integer bit arithmetic, a different mechanism from the
oracle's bit arrays.
"""
import numpy as np
import pytest

from oracle import fp6



def test_decoder_matches_the_format_constants():
    assert fp6.e3m2_decode(0b011111) == 28.0          # largest normal
    assert fp6.e3m2_decode(0b000100) == 0.25          # smallest normal
    assert fp6.e3m2_decode(0b000001) == 0.0625        # smallest subnormal
    assert fp6.e3m2_decode(0b000011) == 0.1875        # largest subnormal
    assert fp6.e3m2_decode(0b001100) == 1.0
    assert fp6.e3m2_decode(0b101100) == -1.0
    assert fp6.e3m2_decode(0b100000) == 0.0           # -0
    # the 32 non-negative codes are strictly increasing (monotone encoding)
    vals = [fp6.e3m2_decode(c) for c in range(32)]
    assert all(a < b for a, b in zip(vals, vals[1:]))


def test_every_4bit_code_is_exact():
    for q in range(-8, 8):
        c = fp6.e3m2_encode(float(q))
        assert 0 <= c < 64
        assert fp6.e3m2_decode(c) == q
    with pytest.raises(ValueError):
        fp6.e3m2_encode(9.0)                           # between 8 and 10: not representable


def test_unpack_int4_nibble_order():
    q4 = np.array([[0x21, 0xF8]], np.uint8)            # k0 = 1, k1 = 2, k2 = -8, k3 = -1
    assert fp6.unpack_int4(q4).tolist() == [[1, 2, -8, -1]]


def test_pack_layout_against_bigint_fields():
    r = np.random.default_rng(6)
    rows, K = 5, 128
    q4 = r.integers(0, 256, size=(rows, K // 2), dtype=np.uint8)
    q6 = fp6.pack_fp6(q4)
    assert q6.shape == (rows, 3 * K // 4) and q6.dtype == np.uint8
    q = fp6.unpack_int4(q4)
    for i in range(rows):
        bits = int.from_bytes(q6[i].tobytes(), "little")
        for k in range(K):
            code = (bits >> (6 * k)) & 63
            assert fp6.e3m2_decode(code) == q[i, k]


def test_single_code_position():
    K = 128
    for k, v in [(0, 1), (1, -8), (5, 7), (127, -1), (64, 3)]:
        q = np.zeros((1, K), np.int16)
        q[0, k] = v
        nib = (q & 0xF).astype(np.uint8)
        q4 = (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)
        q6 = fp6.pack_fp6(q4)
        bits = int.from_bytes(q6[0].tobytes(), "little")
        assert bits == fp6.e3m2_encode(float(v)) << (6 * k)
