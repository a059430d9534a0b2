"""Pins for the oracle's group-decomposed GEMM (APEX4 Sec. 3.2.1,
Eq. group_decomposition):  C = sum_g (A_g^q W_g^q) (.) (S_g^a S_g^w^T).

  * brute force: binary64 GEMM (numpy/BLAS) of the dequantized matrices;
  * unit scales reduce to the exact integer GEMM;
  * G = K reduces to per-channel scaling of the integer GEMM;
  * group merge: P at 2G is the sum of adjacent P at G (exact integers);
  * scales constant along K make the result independent of G (exactly);
  * extremes: all codes -8 give P = 64 G;
  * group sums against numpy's einsum over reshaped groups.
"""
import numpy as np
import pytest

from test_oracle_quant import unpack
from paper_2606_08761_amd import workloads as wl


def dequant(q_packed, scales, G):
    c = unpack(q_packed).astype(np.float64)
    return c * np.repeat(scales.astype(np.float64), G, axis=1)


def rand_case(seed, M, N, K, G):
    r = np.random.default_rng(seed)
    return (wl.random_codes(r, M, K), wl.random_scales(r, M, K // G),
            wl.random_codes(r, N, K), wl.random_scales(r, N, K // G))


SHAPES = [(1, 1, 128, 128), (5, 7, 256, 128), (33, 17, 512, 256), (64, 64, 512, 512),
          (16, 48, 384, 384), (3, 64, 1024, 32), (9, 40, 256, 64)]


@pytest.mark.parametrize("M,N,K,G", SHAPES)
def test_brute_force_dequantized_gemm(O, M, N, K, G):
    Aq, sa, Wq, sw = rand_case(M * 31 + N, M, N, K, G)
    y = O.gemm_rows(Aq, sa, Wq, sw, K, G)
    ref = dequant(Aq, sa, G) @ dequant(Wq, sw, G).T
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


@pytest.mark.parametrize("M,N,K,G", SHAPES)
def test_unit_scales_exact_integer_gemm(O, M, N, K, G):
    Aq, _, Wq, _ = rand_case(M + 7 * N, M, N, K, G)
    ones_a = np.ones((M, K // G), np.float16)
    ones_w = np.ones((N, K // G), np.float16)
    y = O.gemm_rows(Aq, ones_a, Wq, ones_w, K, G)
    exact = unpack(Aq).astype(np.int64) @ unpack(Wq).astype(np.int64).T
    assert np.array_equal(y, exact.astype(np.float64))


@pytest.mark.parametrize("M,N,K", [(4, 6, 256), (17, 9, 1024), (64, 32, 512)])
def test_per_channel_closed_form(O, M, N, K):
    Aq, sa, Wq, sw = rand_case(K + M, M, N, K, K)
    y = O.gemm_rows(Aq, sa, Wq, sw, K, K)
    integer = unpack(Aq).astype(np.int64) @ unpack(Wq).astype(np.int64).T
    ref = sa.astype(np.float64)[:, :1] * sw.astype(np.float64)[:, 0][None, :] * integer
    assert np.array_equal(y, ref)


def test_group_merge_exact(O):
    M, N, K = 12, 20, 1024
    Aq, _, Wq, _ = rand_case(3, M, N, K, 128)
    P = {G: O.groupsums(Aq, Wq, K, G) for G in (32, 64, 128, 256, 512, 1024)}
    for G in (32, 64, 128, 256, 512):
        assert np.array_equal(P[2 * G], P[G][:, :, 0::2] + P[G][:, :, 1::2])
    assert np.array_equal(P[1024][:, :, 0], unpack(Aq).astype(np.int64) @ unpack(Wq).astype(np.int64).T)


def test_groupsums_vs_einsum(O):
    M, N, K, G = 10, 14, 768, 128
    Aq, _, Wq, _ = rand_case(11, M, N, K, G)
    a = unpack(Aq).astype(np.int64).reshape(M, K // G, G)
    w = unpack(Wq).astype(np.int64).reshape(N, K // G, G)
    ref = np.einsum("mgk,ngk->mng", a, w)
    assert np.array_equal(O.groupsums(Aq, Wq, K, G), ref)
    # a row window is the same slice
    assert np.array_equal(O.groupsums(Aq, Wq, K, G, m0=3, mr=4), ref[3:7])


def test_constant_scales_independent_of_G(O):
    M, N, K = 9, 11, 1024
    r = np.random.default_rng(12)
    Aq = wl.random_codes(r, M, K)
    Wq = wl.random_codes(r, N, K)
    alpha = wl.random_scales(r, M, 1)
    beta = wl.random_scales(r, N, 1)
    ys = []
    for G in (32, 128, 256, 1024):
        sa = np.repeat(alpha, K // G, axis=1)
        sw = np.repeat(beta, K // G, axis=1)
        ys.append(O.gemm_rows(Aq, sa, Wq, sw, K, G))
    for y in ys[1:]:
        assert np.array_equal(y, ys[0])


@pytest.mark.parametrize("G", [32, 128, 512])
def test_extremes(O, G):
    M, N, K = 3, 5, 1024
    neg8 = np.full((M, K // 2), 0x88, np.uint8)        # every code -8
    pos7 = np.full((N, K // 2), 0x77, np.uint8)        # every code 7
    P = O.groupsums(neg8, np.full((N, K // 2), 0x88, np.uint8), K, G)
    assert (P == 64 * G).all()
    P = O.groupsums(neg8, pos7, K, G)
    assert (P == -56 * G).all()
    ones_a = np.ones((M, K // G), np.float16)
    ones_w = np.ones((N, K // G), np.float16)
    neg8_w = np.full((N, K // 2), 0x88, np.uint8)
    assert (O.gemm_rows(neg8, ones_a, neg8_w, ones_w, K, G) == 64.0 * K).all()


def test_row_subset_and_f16_output(O):
    M, N, K, G = 40, 24, 512, 128
    Aq, sa, Wq, sw = rand_case(21, M, N, K, G)
    full = O.gemm_rows(Aq, sa, Wq, sw, K, G)
    rows = np.array([39, 0, 17, 17, 5])
    assert np.array_equal(O.gemm_rows(Aq, sa, Wq, sw, K, G, rows), full[rows])
    Y = O.gemm_f16(Aq, sa, Wq, sw, K, G)
    assert np.array_equal(Y.view(np.uint16), full.astype(np.float16).view(np.uint16))


def test_transposed_operands_are_distinguished(O):
    """Y = A W^T: swapping the roles of A and W transposes the output."""
    M, N, K, G = 6, 9, 256, 128
    Aq, sa, Wq, sw = rand_case(33, M, N, K, G)
    y = O.gemm_rows(Aq, sa, Wq, sw, K, G)
    yt = O.gemm_rows(Wq, sw, Aq, sa, K, G)
    assert np.array_equal(y.T, yt)
