"""GPU parity of the split-K GEMM (apex4_w4a4_gemm_ws; APEX4 Eq.
group_decomposition summed over K ranges of whole groups, then over ranges),
for G = 128 (the ping-pong kernel) and the other group sizes (the general tile
kernel; per-channel partials are exact, so that split is bit-identical).

  * where a split applies, Y is within |Y - y| <= 2e-3 |y| + 1e-2 RMS_row(y)
    of the oracle's binary64 y, and two calls give the same bits;
  * where none applies (workspace size 0), Y is apex4_w4a4_gemm's, bit for bit;
  * a missing or short workspace is refused with APEX4_ERR_WORKSPACE.
"""
import numpy as np
import pytest

from parity import check_tolerance, dev, host, log, sample_rows
from paper_2606_08761_amd import workloads as wl

pytestmark = pytest.mark.gpu

G = 128


def pk():
    import paper_2606_08761_amd as m
    return m


def operands(M, N, K, seed):
    r = np.random.default_rng(seed)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    return Aq, sa, Wq, sw


# (M, N, K): split factors 8, 4 and 2, ragged tiles (M = 260: a 4-row tile),
# odd M N (the reduction's one-element path), 4 stages per split
SPLIT = [(33, 8192, 8192), (64, 8192, 8192), (256, 8192, 8192), (512, 8192, 4096), (100, 1000, 2048),
         (130, 4100, 2048), (65, 1001, 2048), (200, 2000, 2048), (260, 6144, 8192)]


@pytest.mark.parametrize("M,N,K", SPLIT)
def test_split_matches_oracle(O, M, N, K):
    m = pk()
    need = m.apex4_w4a4_gemm_workspace_size(M, N, K, G)
    log(f"split-K M={M} N={N} K={K} workspace={need}")
    assert need > 0 and need % (4 * M * N) == 0 and need // (4 * M * N) in (2, 4, 8)
    Aq, sa, Wq, sw = operands(M, N, K, M * 131 + N + K)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    import torch
    ws = torch.empty((need,), dtype=torch.uint8, device="cuda")
    Y1 = host(m.apex4_w4a4_gemm_ws(*d, G, ws))
    Y2 = host(m.apex4_w4a4_gemm_ws(*d, G, ws))
    assert np.array_equal(Y1.view(np.uint16), Y2.view(np.uint16))
    rows = sample_rows(M, seed=M) if M > 64 else np.arange(M)
    check_tolerance(Y1[rows], O.gemm_rows(Aq, sa, Wq, sw, K, G, rows), f"split-K {M}x{N}x{K}")


@pytest.mark.parametrize("M,N,K,GG", [(2048, 8192, 1024, 128), (16, 8192, 1024, 128), (1, 4096, 1024, 128),
                                      (256, 8192, 1024, 64), (256, 8192, 1024, 1024), (64, 1024, 384, 128),
                                      (64, 28672, 1024, 128)])
def test_no_split_is_the_plain_gemm(M, N, K, GG):
    """No workspace needed: the same kernels as apex4_w4a4_gemm run (K = 384 has
    too few stages per split; with G != 128 at M = 256, N = 8192 the small tiles
    already fill the CUs; M = 64 with N = 28672 would only split in two)."""
    m = pk()
    assert m.apex4_w4a4_gemm_workspace_size(M, N, K, GG) == 0
    r = np.random.default_rng(M + N + K + GG)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // GG), wl.random_scales(r, N, K // GG)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    Y0 = host(m.apex4_w4a4_gemm(*d, GG))
    Yw = host(m.apex4_w4a4_gemm_ws(*d, GG))
    assert np.array_equal(Y0.view(np.uint16), Yw.view(np.uint16))


def test_workspace_refused_when_short():
    import torch
    m = pk()
    M, N, K = 64, 8192, 8192
    need = m.apex4_w4a4_gemm_workspace_size(M, N, K, G)
    Aq, sa, Wq, sw = operands(M, N, K, 5)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    short = torch.empty((need - 16,), dtype=torch.uint8, device="cuda")
    with pytest.raises(m.Apex4Error) as e:
        m.apex4_w4a4_gemm_ws(*d, G, short)
    assert e.value.status == -7


# the general tile kernel split over K: fine groups, persisting groups (splits
# on group boundaries), per-channel (exact int32 partials)
SPLIT_G = [(256, 1024, 8192, 32), (128, 2048, 4096, 64), (200, 1000, 4096, 256), (100, 1000, 2048, 1024),
           (65, 1001, 2048, 32), (64, 2048, 8192, 8192), (300, 520, 3072, 3072)]


@pytest.mark.parametrize("M,N,K,GG", SPLIT_G)
def test_split_other_groups(O, M, N, K, GG):
    import torch
    m = pk()
    need = m.apex4_w4a4_gemm_workspace_size(M, N, K, GG)
    log(f"split-K M={M} N={N} K={K} G={GG} workspace={need}")
    assert need > 0 and need // (4 * M * N) in (2, 4, 8)
    r = np.random.default_rng(M * 7 + N + K + GG)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // GG), wl.random_scales(r, N, K // GG)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    ws = torch.empty((need,), dtype=torch.uint8, device="cuda")
    Y1 = host(m.apex4_w4a4_gemm_ws(*d, GG, ws))
    Y2 = host(m.apex4_w4a4_gemm_ws(*d, GG, ws))
    assert np.array_equal(Y1.view(np.uint16), Y2.view(np.uint16))
    if GG == K:
        # per-channel partial sums are exact integers: the split changes no bit
        Y0 = host(m.apex4_w4a4_gemm(*d, GG))
        assert np.array_equal(Y1.view(np.uint16), Y0.view(np.uint16))
    rows = sample_rows(M, seed=M) if M > 64 else np.arange(M)
    check_tolerance(Y1[rows], O.gemm_rows(Aq, sa, Wq, sw, K, GG, rows), f"split-K {M}x{N}x{K} G{GG}")
