"""Reduction lengths that are not a multiple of the 128-wide K stage.

The boundary takes any K >= 32 with K % 32 == 0 (and K % G == 0).  With
G in {32, 64} or G == K the kernels' last K stage is then partial: its missing
codes load as zeros and its missing groups are skipped.  Checked against the
oracle through every entry point that takes K:

  * apex4_quantize_act: codes and scales bit-exact, including group sizes that
    are neither a power of two nor K (G = 96, 160);
  * apex4_w4a4_gemm: exact group sums (debug dump, same launches as Y) and Y
    within tolerance, on the one-row, few-row and both tile kernels;
  * apex4_w4a4_gemm_ws: the split over K with a partial last stage;
  * apex4_w4a4_linear: Y and work buffers equal quantize-then-GEMM bit for bit;
  * the largest per-channel K (65536) with extreme codes, where 256 P reaches
    2^30 in the kernels' int32 sums.
"""
import numpy as np
import pytest

from parity import check_tolerance, dev, host, log
from paper_2606_08761_amd import workloads as wl

pytestmark = pytest.mark.gpu

# (K, G): K % 128 != 0 except where noted
KG = [(32, 32), (96, 32), (96, 96), (160, 32), (160, 160), (192, 64), (8224, 32), (8224, 8224), (8256, 64),
      (4000, 32)]


def pk():
    import paper_2606_08761_amd as m
    return m


@pytest.mark.parametrize("K,G", KG + [(96 * 5, 96), (160 * 3, 160), (96 * 64, 96), (8224, 8224)])
def test_quantize_k_tail(O, K, G):
    m = pk()
    M = 37
    x = wl.activations(wl.rng_for("tiny", 40, K + G), M, K)
    q, s = m.apex4_quantize_act(dev(x), G)
    q_o, s_o = O.quantize(x, G)
    assert np.array_equal(host(q), q_o), (K, G)
    assert np.array_equal(host(s).view(np.uint16), s_o.view(np.uint16)), (K, G)


# (M, N): one row, the streaming kernel, the 64 x 128 tiles (with and without the
# in-workgroup K split), the 128 x 256 tiles
MN = [(1, 520), (7, 40), (32, 300), (100, 136), (300, 520), (2048, 4096)]


@pytest.mark.parametrize("M,N", MN)
@pytest.mark.parametrize("K,G", KG)
def test_gemm_k_tail(O, M, N, K, G):
    import torch
    m = pk()
    plan = m.apex4_w4a4_gemm_plan("gemm", M, N, K, G)
    log(f"k tail gemm M={M} N={N} K={K} G={G}: {plan}")
    r = np.random.default_rng(M * 7 + N * 11 + K * 13 + G)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    Y = m.apex4_w4a4_gemm(*d, G)
    m0, mr = (0, M) if M <= 300 else (126, 4)
    Yd, P = m.apex4_w4a4_gemm_debug(*d, G, m0, mr)
    torch.cuda.synchronize()
    assert torch.equal(Yd, Y)
    assert np.array_equal(host(P), O.groupsums(Aq, Wq, K, G, m0, mr))
    rows = np.arange(M) if M <= 300 else np.concatenate([np.arange(0, 4), np.arange(126, 130), np.arange(M - 4, M)])
    check_tolerance(host(Y)[rows], O.gemm_rows(Aq, sa, Wq, sw, K, G, rows), f"k tail {M}x{N}x{K} G{G}")


# split over K with a partial last stage: 128 stages, the last holding 32 of 128 codes
SPLIT = [(128, 1024, 16352, 32), (128, 1024, 16352, 16352), (256, 2048, 16352, 32)]


@pytest.mark.parametrize("M,N,K,G", SPLIT)
def test_gemm_ws_k_tail(O, M, N, K, G):
    import torch
    m = pk()
    kern, S = m.apex4_w4a4_gemm_plan("gemm_ws", M, N, K, G)
    log(f"k tail split M={M} N={N} K={K} G={G}: {kern} S={S}")
    assert S > 1
    need = m.apex4_w4a4_gemm_workspace_size(M, N, K, G)
    assert need == S * M * N * 4
    r = np.random.default_rng(M + N + K + G)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    ws = torch.empty((need,), dtype=torch.uint8, device="cuda")
    Y = m.apex4_w4a4_gemm_ws(*d, G, ws)
    Yd, P = m.apex4_w4a4_gemm_debug(*d, G, 60, 8, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(Yd, Y)
    assert np.array_equal(host(P), O.groupsums(Aq, Wq, K, G, 60, 8))
    rows = np.arange(0, M, 7)
    check_tolerance(host(Y)[rows], O.gemm_rows(Aq, sa, Wq, sw, K, G, rows), f"k tail split {M}x{N}x{K}")
    if G == K:  # the per-channel split sums exact integers: the same bits as unsplit
        assert torch.equal(Y, m.apex4_w4a4_gemm(*d, G))


@pytest.mark.parametrize("M", [1, 5, 100])
@pytest.mark.parametrize("K,G", [(96, 32), (160, 32), (192, 64), (8224, 32), (8224, 8224), (4000, 32)])
def test_linear_k_tail(O, M, K, G):
    import torch
    m = pk()
    N = 264
    plan = m.apex4_w4a4_gemm_plan("linear", M, N, K, G)
    log(f"k tail linear M={M} K={K} G={G}: {plan}")
    x = wl.activations(wl.rng_for("decode", 41, M * 7 + K + G), M, K)
    w = wl.weights(wl.rng_for("decode", 42, K + G), N, K)
    Wq_d, sw_d = m.apex4_quantize_act(dev(w), G)
    Aw = torch.full((M, K // 2), 0xAB, dtype=torch.uint8, device="cuda")
    sw_ = torch.full((M, K // G), float("nan"), dtype=torch.float16, device="cuda")
    Y = m.apex4_w4a4_linear(dev(x), Wq_d, sw_d, G, A_q_work=Aw, s_a_work=sw_)
    Aq_d, sa_d = m.apex4_quantize_act(dev(x), G)
    Y2 = m.apex4_w4a4_gemm(Aq_d, sa_d, Wq_d, sw_d, G)
    torch.cuda.synchronize()
    assert torch.equal(Aw, Aq_d) and torch.equal(sw_.view(torch.int16), sa_d.view(torch.int16))
    assert torch.equal(Y, Y2)
    Wq_o, sw_o = O.quantize(w, G)
    Aq_o, sa_o = O.quantize(x, G)
    assert np.array_equal(host(Wq_d), Wq_o) and np.array_equal(host(Aq_d), Aq_o)
    check_tolerance(host(Y), O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G), f"k tail linear {M}x{K} G{G}")
    Yl, _, _, P = m.apex4_w4a4_linear_debug(dev(x), Wq_d, sw_d, G)
    torch.cuda.synchronize()
    assert torch.equal(Yl, Y)
    assert np.array_equal(host(P), O.groupsums(Aq_o, Wq_o, K, G))


@pytest.mark.parametrize("M", [1, 8, 64, 300])
def test_largest_channel_k_extreme_codes(O, M):
    """G = K = 65536 with every code -8 (and 7 on even weight rows): |P| = 2^22,
    the kernels' int32 holds 256 P = 2^30."""
    import torch
    m = pk()
    N, K = 72, 65536
    G = K
    Aq = np.full((M, K // 2), 0x88, np.uint8)
    Wq = np.full((N, K // 2), 0x88, np.uint8)
    Wq[::2] = 0x77
    s_a = np.full((M, 1), 2.0 ** -10, np.float16)
    s_w = np.full((N, 1), 2.0 ** -10, np.float16)
    d = [dev(a) for a in (Aq, s_a, Wq, s_w)]
    P_o = O.groupsums(Aq, Wq, K, G)
    assert P_o.max() == 2 ** 22 and P_o.min() == -56 * K
    y = O.gemm_rows(Aq, s_a, Wq, s_w, K, G)
    for entry in ("gemm", "gemm_ws"):
        plan = m.apex4_w4a4_gemm_plan(entry, M, N, K, G)
        log(f"largest channel K M={M} {entry}: {plan}")
        ws = None
        if entry == "gemm_ws":
            ws = torch.empty((max(m.apex4_w4a4_gemm_workspace_size(M, N, K, G), 16),), dtype=torch.uint8,
                             device="cuda")
        Yd, P = m.apex4_w4a4_gemm_debug(*d, G, workspace=ws)
        torch.cuda.synchronize()
        assert np.array_equal(host(P), P_o), entry
        check_tolerance(host(Yd), y, f"largest channel K M={M} {entry}")
