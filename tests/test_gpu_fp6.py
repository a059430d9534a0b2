"""GPU parity of the FP6-container W4A4 GEMM (APEX4 Sec. 3.2.1, Eq.
group_decomposition, on the f8f6f4 matrix cores of gfx950).

  * apex4_pack_fp6 is bit-identical to the oracle's e3m2 re-encoding;
  * apex4_w4a4_gemm_fp6 on the re-encoded codes returns the same bits as
    apex4_w4a4_gemm on the 4-bit codes wherever that runs its 128 x 256 tile
    kernel (same operation order: M > 32 and at least one tile per compute
    unit; smaller problems go to kernels that split K), and is always within
    |Y - y| <= 2e-3 |y| + 1e-2 RMS_row(y) of the oracle's binary64 y;
  * shapes: tiny, ragged (partial tiles, odd N, odd stage counts), extreme
    codes, the M=2048 N=K=8192 shape on sampled rows.
"""
import numpy as np
import pytest

from oracle import fp6 as ofp6
from parity import check_tolerance, dev, host, log, sample_rows
from paper_2606_08761_amd import workloads as wl

pytestmark = pytest.mark.gpu

G = 128


def pk():
    import paper_2606_08761_amd as m
    return m


def both(Aq, sa, Wq, sw):
    """(Y from the FP6 GEMM, Y from the INT8-core GEMM), packing on the device."""
    m = pk()
    A6, W6 = m.apex4_pack_fp6(dev(Aq)), m.apex4_pack_fp6(dev(Wq))
    sa_d, sw_d = dev(sa), dev(sw)
    Y6 = host(m.apex4_w4a4_gemm_fp6(A6, sa_d, W6, sw_d, G))
    Y4 = host(m.apex4_w4a4_gemm(dev(Aq), sa_d, dev(Wq), sw_d, G))
    return Y6, Y4


def same_order_as_int4(M, N):
    """apex4_w4a4_gemm runs the 128 x 256 tile kernel for this shape."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    return M > 32 and ((M + 127) // 128) * ((N + 255) // 256) >= cus


def check_same_bits(Y6, Y4, M, N):
    if same_order_as_int4(M, N):
        assert np.array_equal(Y6.view(np.uint16), Y4.view(np.uint16))


def test_pack_matches_oracle():
    r = np.random.default_rng(66)
    for rows, K in ((1, 128), (37, 384), (300, 1152), (1024, 8192)):
        log(f"pack rows={rows} K={K}")
        q4 = r.integers(0, 256, size=(rows, K // 2), dtype=np.uint8)
        q6 = host(pk().apex4_pack_fp6(dev(q4)))
        assert np.array_equal(q6, ofp6.pack_fp6(q4)), (rows, K)


def test_tiny_full(O):
    M, N, K = 64, 1024, 1024
    log("fp6 tiny")
    Aq, sa, Wq, sw = wl.codes_workload("tiny", M, N, K, G)
    Y6, Y4 = both(Aq, sa, Wq, sw)
    check_same_bits(Y6, Y4, M, N)
    check_tolerance(Y6, O.gemm_rows(Aq, sa, Wq, sw, K, G), "fp6 tiny")


RAGGED = [(1, 1, 128), (8, 200, 256), (300, 260, 384), (129, 136, 512), (255, 257, 768),
          (1111, 8200, 640), (1500, 8195, 1152), (2050, 4100, 4096)]


@pytest.mark.parametrize("M,N,K", RAGGED)
def test_ragged(O, M, N, K):
    log(f"fp6 ragged M={M} N={N} K={K}")
    r = np.random.default_rng(M * 7919 + N * 31 + K + 6)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    Y6, Y4 = both(Aq, sa, Wq, sw)
    check_same_bits(Y6, Y4, M, N)
    rows = sample_rows(M, seed=M) if M > 64 else np.arange(M)
    check_tolerance(Y6[rows], O.gemm_rows(Aq, sa, Wq, sw, K, G, rows), f"fp6 ragged {M}x{N}x{K}")


@pytest.mark.parametrize("code", [-8, 7])
def test_extreme_codes(O, code):
    """Every product at its largest magnitude (64 or 49): group sums of 8192 or 6272."""
    M, N, K = 2048, 4096, 1024
    log(f"fp6 extreme codes {code}")
    nib = np.uint8(code & 0xF)
    Aq = np.full((M, K // 2), nib | (nib << 4), np.uint8)
    Wq = np.full((N, K // 2), nib | (nib << 4), np.uint8)
    r = np.random.default_rng(8)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    Y6, Y4 = both(Aq, sa, Wq, sw)
    check_same_bits(Y6, Y4, M, N)
    check_tolerance(Y6, O.gemm_rows(Aq, sa, Wq, sw, K, G), f"fp6 extreme {code}")


def test_paper_shape_sampled(O):
    M, N, K = 2048, 8192, 8192
    log("fp6 paper shape")
    Aq, sa, Wq, sw = wl.codes_workload("paper", M, N, K, G)
    Y6, Y4 = both(Aq, sa, Wq, sw)
    assert same_order_as_int4(M, N)
    check_same_bits(Y6, Y4, M, N)
    rows = sample_rows(M, seed=11)
    check_tolerance(Y6[rows], O.gemm_rows(Aq, sa, Wq, sw, K, G, rows), "fp6 paper shape")


def test_empty_and_group_rule():
    m = pk()
    import torch
    A6 = torch.empty((0, 96), dtype=torch.uint8, device="cuda")
    sa = torch.empty((0, 1), dtype=torch.float16, device="cuda")
    W6 = torch.zeros((8, 96), dtype=torch.uint8, device="cuda")
    sw = torch.zeros((8, 1), dtype=torch.float16, device="cuda")
    assert m.apex4_w4a4_gemm_fp6(A6, sa, W6, sw, G).shape == (0, 8)
    with pytest.raises(m.Apex4Error):
        m.apex4_w4a4_gemm_fp6(A6, sa, W6, sw, 64)
