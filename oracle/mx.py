"""Power-of-two (E8M0) group scales: the MX numerics variant (test infrastructure only).

Only the tests may import this module; the product library never does.

APEX4's SymQuant (Sec. 3.2.1, Eq. SymQuant) takes the group scale
S = max|X_g| / 7 in FP16.  This variant keeps the 4-bit symmetric codes and the
groups but restricts S to a power of two, 2^E, the smallest one that still
covers the group: E = min{ e integer : max|X_g| <= 7 * 2^e }.  Such scales can
be applied inside a block-scaled matrix instruction, so the per-group
dequantization the paper identifies as the bottleneck disappears (the paper
notes that FP4 with folded block scaling needs no separate dequantization,
Sec. 2.2).  The scale is stored as an E8M0 byte, E + 127.

  * codes: q = clamp(round_half_even(x / 2^E), -8, 7), |q| <= 7 by the choice of E;
  * a group with max|X_g| = 0 stores E = 0 (byte 127) and zero codes;
  * GEMM: Y[m,n] = binary16( sum_g 2^(E_a[m,g] + E_w[n,g]) P[m,n,g] ),
    P as in Eq. (group_decomposition); every term is exact in binary64, the
    terms are summed in binary64 and the sum is rounded once.

Codes are returned packed like the fp16-scale quantizer's ([rows, K/2] uint8,
low nibble = even k); oracle.fp6.pack_fp6 re-encodes them as FP6 containers.
"""
from __future__ import annotations

import math

import numpy as np


def group_exponent(amax: float) -> int:
    """Smallest integer e with amax <= 7 * 2^e (0 for amax == 0)."""
    if amax == 0:
        return 0
    e = math.ceil(math.log2(amax / 7.0))
    # log2 of a float quotient can land one off; settle it exactly
    while amax > 7.0 * 2.0 ** e:
        e += 1
    while amax <= 7.0 * 2.0 ** (e - 1):
        e -= 1
    return e


def quantize_mx(x: np.ndarray, G: int):
    """x binary16 [M, K] -> (codes uint8 [M, K/2] packed, e8m0 uint8 [M, K/G])."""
    x = np.asarray(x, np.float16)
    M, K = x.shape
    if K % G:
        raise ValueError("K % G != 0")
    xf = x.astype(np.float64).reshape(M, K // G, G)
    amax = np.abs(xf).max(axis=2)
    E = np.vectorize(group_exponent, otypes=[np.int64])(amax)
    q = np.rint(xf / np.exp2(E)[:, :, None])           # exact quotient (power of two), ties to even
    q = np.clip(q, -8, 7).astype(np.int16).reshape(M, K)
    nib = (q & 0xF).astype(np.uint8)
    codes = (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)
    return codes, (E + 127).astype(np.uint8)


def unpack(codes: np.ndarray) -> np.ndarray:
    lo = (codes & 0xF).astype(np.int64)
    hi = (codes >> 4).astype(np.int64)
    q = np.empty((codes.shape[0], 2 * codes.shape[1]), np.int64)
    q[:, 0::2], q[:, 1::2] = lo, hi
    return np.where(q >= 8, q - 16, q)


def gemm_mx(Aq, ea, Wq, ew, K: int, G: int, rows=None) -> np.ndarray:
    """Y rows (binary16) of the MX GEMM; rows = None for all of them."""
    y = gemm_mx_f64(Aq, ea, Wq, ew, K, G, rows)
    with np.errstate(over="ignore"):      # beyond the binary16 range: +-inf, as the rounding defines
        return y.astype(np.float16)


def gemm_mx_f64(Aq, ea, Wq, ew, K: int, G: int, rows=None) -> np.ndarray:
    """The binary64 sum of the MX GEMM before its final rounding."""
    A = unpack(np.asarray(Aq))
    W = unpack(np.asarray(Wq))
    if rows is not None:
        A, ea = A[rows], np.asarray(ea)[rows]
    ng = K // G
    y = np.zeros((A.shape[0], W.shape[0]), np.float64)
    for g in range(ng):
        P = A[:, g * G:(g + 1) * G] @ W[:, g * G:(g + 1) * G].T          # exact int64
        s = np.exp2(ea[:, g].astype(np.float64) - 127)[:, None] * np.exp2(ew[:, g].astype(np.float64) - 127)[None, :]
        y += s * P                                                       # each term exact: power of two times integer
    return y
