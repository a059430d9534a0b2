"""FP6 e3m2 containers for 4-bit codes (test infrastructure only).

Only the tests may import this module; the product library never does.

A code q in [-8, 7] of Eq. (SymQuant) (APEX4 Sec. 3.2.1) is stored in the
6-bit e3m2 format of the OCP Microscaling formats (1 sign bit, 3 exponent bits
with bias 3, 2 mantissa bits, no infinities or NaN): normal values
(-1)^s 2^(e-3) (1 + m/4) for e > 0, subnormal values (-1)^s 2^-2 (m/4) for
e = 0.  The row layout is the library's FP6 layout: code k of a row in bits
[6k, 6k + 6) of the row's bytes read as one little-endian bit string.

The encoder searches every one of the 64 codes for the one that decodes to the
wanted value, so it is only as good as the decoder, which is the format's
definition written out.
"""
from __future__ import annotations

import numpy as np


def e3m2_decode(code: int) -> float:
    """Value of a 6-bit e3m2 code."""
    s, e, m = (code >> 5) & 1, (code >> 2) & 7, code & 3
    mag = 2.0 ** -2 * (m / 4) if e == 0 else 2.0 ** (e - 3) * (1 + m / 4)
    return -mag if s else mag


def e3m2_encode(v: float) -> int:
    """The e3m2 code whose value is exactly v (+0 for zero); ValueError if none."""
    if v == 0:
        return 0
    hits = [c for c in range(64) if e3m2_decode(c) == v]
    if len(hits) != 1:
        raise ValueError(f"{v} is not exactly representable in e3m2")
    return hits[0]


def unpack_int4(q4: np.ndarray) -> np.ndarray:
    """Packed codes uint8 [rows, K/2] (low nibble = even k) -> int8 [rows, K]."""
    q4 = np.asarray(q4, np.uint8)
    lo = (q4 & 0xF).astype(np.int16)
    hi = (q4 >> 4).astype(np.int16)
    out = np.empty((q4.shape[0], 2 * q4.shape[1]), np.int16)
    out[:, 0::2], out[:, 1::2] = lo, hi
    return np.where(out >= 8, out - 16, out).astype(np.int8)


def pack_fp6(q4: np.ndarray) -> np.ndarray:
    """Packed 4-bit codes uint8 [rows, K/2] -> e3m2 codes uint8 [rows, 3K/4]."""
    q = unpack_int4(q4)
    table = np.array([e3m2_encode(float(v)) for v in range(-8, 8)], np.uint8)
    codes = table[q.astype(np.int16) + 8]
    rows, K = codes.shape
    bits = ((codes[:, :, None] >> np.arange(6, dtype=np.uint8)) & 1).reshape(rows, 6 * K)
    return np.packbits(bits, axis=1, bitorder="little")
