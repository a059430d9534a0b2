"""Pins of the MX-variant oracle (oracle/mx.py), CPU only.

The power-of-two scale is pinned by its defining inequality at exact
boundaries and by a hand-worked group; the codes by the rounding rule and the
error bound; the GEMM by brute force over the dequantized matrices, by unit
scales (the integer GEMM), by the scale algebra (a common exponent shift scales
Y by that power of two) and by the fp16-scale GEMM of the same codes when
every scale is 1.
"""
import numpy as np
import pytest

from oracle import mx


def test_exponent_boundaries():
    assert mx.group_exponent(7.0) == 0                    # amax = 7 * 2^0 exactly: E = 0
    assert mx.group_exponent(float(np.nextafter(7.0, 8.0))) == 1
    assert mx.group_exponent(3.5) == -1
    assert mx.group_exponent(28.0) == 2
    assert mx.group_exponent(28.01) == 3
    assert mx.group_exponent(65504.0) == 14               # largest fp16
    assert mx.group_exponent(2.0 ** -24) == -26           # smallest fp16 subnormal
    assert mx.group_exponent(0.0) == 0
    for e in range(-20, 12):
        a = 7.0 * 2.0 ** e
        assert mx.group_exponent(a) == e and mx.group_exponent(a * 1.0001) == e + 1


def test_worked_group():
    # amax 5.0 -> E = 0 (5 <= 7); x / 1 rounded half to even: 2.5 -> 2, -3.5 -> -4, 0.5 -> 0
    x = np.zeros((1, 32), np.float16)
    x[0, :6] = [5.0, 2.5, -3.5, 0.5, -1.25, 1.75]
    codes, e = mx.quantize_mx(x, 32)
    q = mx.unpack(codes)[0]
    assert e.tolist() == [[127]]
    assert q[:6].tolist() == [5, 2, -4, 0, -1, 2] and not q[6:].any()
    # amax 14 -> E = 1: codes x / 2
    x2 = np.zeros((1, 32), np.float16)
    x2[0, :3] = [14.0, -3.0, 1.0]
    c2, e2 = mx.quantize_mx(x2, 32)
    assert e2.tolist() == [[128]] and mx.unpack(c2)[0, :3].tolist() == [7, -2, 0]   # -1.5 -> -2, 0.5 -> 0


def test_codes_bound_and_error():
    r = np.random.default_rng(1)
    x = (r.standard_normal((16, 512)) * np.exp2(r.integers(-10, 6, size=(16, 1)))).astype(np.float16)
    for G in (32, 64, 128, 512):
        codes, e = mx.quantize_mx(x, G)
        q = mx.unpack(codes)
        assert np.abs(q).max() <= 7
        s = np.repeat(np.exp2(e.astype(np.float64) - 127), G, axis=1)
        err = np.abs(x.astype(np.float64) - q * s)
        assert (err <= s / 2).all()
        # the scale is the smallest power of two that covers the group
        amax = np.abs(x.astype(np.float64)).reshape(16, -1, G).max(axis=2)
        assert (amax <= 7 * np.exp2(e - 127.0)).all() and (amax > 7 * np.exp2(e - 128.0)).all()


def test_zero_group():
    codes, e = mx.quantize_mx(np.zeros((2, 64), np.float16), 32)
    assert not codes.any() and (e == 127).all()


def _random_codes(r, rows, K):
    return r.integers(0, 256, size=(rows, K // 2), dtype=np.uint8)


def test_gemm_brute_force():
    r = np.random.default_rng(2)
    M, N, K, G = 5, 7, 256, 64
    Aq, Wq = _random_codes(r, M, K), _random_codes(r, N, K)
    ea = (127 + r.integers(-8, 3, size=(M, K // G))).astype(np.uint8)
    ew = (127 + r.integers(-8, 3, size=(N, K // G))).astype(np.uint8)
    A = mx.unpack(Aq) * np.repeat(np.exp2(ea - 127.0), G, axis=1)
    W = mx.unpack(Wq) * np.repeat(np.exp2(ew - 127.0), G, axis=1)
    ref = np.array([[sum(float(A[m, k]) * float(W[n, k]) for k in range(K)) for n in range(N)] for m in range(M)])
    assert np.array_equal(mx.gemm_mx(Aq, ea, Wq, ew, K, G), ref.astype(np.float16))


def test_gemm_unit_scales_and_shift():
    r = np.random.default_rng(3)
    M, N, K, G = 6, 9, 512, 128
    Aq, Wq = _random_codes(r, M, K), _random_codes(r, N, K)
    one_a = np.full((M, K // G), 127, np.uint8)
    one_w = np.full((N, K // G), 127, np.uint8)
    P = mx.unpack(Aq) @ mx.unpack(Wq).T
    assert np.array_equal(mx.gemm_mx(Aq, one_a, Wq, one_w, K, G), P.astype(np.float16))
    # moving 3 binary orders from the activation scales to the weight scales
    # leaves Y unchanged; a shift of A's scales alone by -3 divides it by 8
    # (exact away from the fp16 subnormal range)
    ea = (127 + r.integers(-4, 4, size=(M, K // G))).astype(np.uint8)
    ew = (127 + r.integers(-4, 4, size=(N, K // G))).astype(np.uint8)
    y0 = mx.gemm_mx(Aq, ea, Wq, ew, K, G).astype(np.float64)
    assert np.array_equal(mx.gemm_mx(Aq, ea + 3, Wq, ew - 3, K, G).astype(np.float64), y0)
    y3 = mx.gemm_mx(Aq, ea - 3, Wq, ew, K, G).astype(np.float64)
    normal = np.abs(y0) >= 2.0 ** -11
    assert np.array_equal(y3[normal] * 8, y0[normal])
    # row subset
    rows = np.array([4, 0, 2])
    assert np.array_equal(mx.gemm_mx(Aq, ea, Wq, ew, K, G, rows), mx.gemm_mx(Aq, ea, Wq, ew, K, G)[rows])


def test_gemm_matches_fp16_scale_gemm_at_unit_scales(O):
    """With every scale 1 the MX GEMM and the fp16-scale GEMM of the same codes coincide."""
    r = np.random.default_rng(4)
    M, N, K, G = 4, 8, 256, 128
    Aq, Wq = _random_codes(r, M, K), _random_codes(r, N, K)
    ones = lambda rows: np.ones((rows, K // G), np.float16)
    y16 = O.gemm_f16(Aq, ones(M), Wq, ones(N), K, G)
    ymx = mx.gemm_mx(Aq, np.full((M, K // G), 127, np.uint8), Wq, np.full((N, K // G), 127, np.uint8), K, G)
    assert np.array_equal(y16.view(np.uint16), ymx.view(np.uint16))
