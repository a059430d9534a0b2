"""The offline tiled weight layout (apex4_tile_weights) and the GEMM and linear
entry points that read it.

  * the layout itself, against its definition written out on the host:
    W_t[t][s][j][l][b] = W_q[32 t + l % 32][64 s + 32 (l / 32) + 16 j + b],
    zero past N and K/2 (ragged N and K included);
  * Y from tiled weights equals Y from row-major weights bit for bit on every
    kernel that reads the same lane fragments (streaming, both tile kernels,
    ping-pong, split over K), and is within tolerance of the oracle on one or
    two rows (the dot-product kernel adds its partial sums in another order);
  * exact group sums through the tiled paths (debug dump) against the oracle;
  * the linear entry point: Y and work buffers equal quantize-then-GEMM.
"""
import numpy as np
import pytest

from parity import check_tolerance, dev, host, log
from paper_2606_08761_amd import workloads as wl

pytestmark = pytest.mark.gpu


def pk():
    import paper_2606_08761_amd as m
    return m


def tiled_reference(Wq: np.ndarray) -> np.ndarray:
    """The tiled layout by its definition, one 16-byte piece at a time."""
    N, kb = Wq.shape
    T, S = -(-N // 32), -(-kb // 64)
    out = np.zeros((T, S, 2, 64, 16), np.uint8)
    for t in range(T):
        for s in range(S):
            for j in range(2):
                for l in range(64):
                    row, b0 = 32 * t + l % 32, 64 * s + 32 * (l // 32) + 16 * j
                    if row < N and b0 < kb:
                        out[t, s, j, l] = Wq[row, b0:b0 + 16]
    return out.reshape(-1)


@pytest.mark.parametrize("N,K", [(32, 128), (40, 256), (100, 160), (64, 8224), (33, 96)])
def test_tiled_layout_definition(N, K):
    m = pk()
    r = np.random.default_rng(N * 3 + K)
    Wq = wl.random_codes(r, N, K)
    assert m.apex4_tiled_weights_size(N, K) == -(-N // 32) * -(-K // 128) * 2048
    Wt = host(m.apex4_tile_weights(dev(Wq)))
    assert np.array_equal(Wt, tiled_reference(Wq))


def test_tiled_layout_large():
    """A Llama-2-70B-sized matrix: spot pieces against the definition."""
    m = pk()
    N, K = 8200, 8192
    r = np.random.default_rng(11)
    Wq = wl.random_codes(r, N, K)
    Wt = host(m.apex4_tile_weights(dev(Wq))).reshape(-(-N // 32), K // 128, 2, 64, 16)
    for t, s, j, l in zip(r.integers(0, Wt.shape[0], 64), r.integers(0, K // 128, 64), r.integers(0, 2, 64),
                          r.integers(0, 64, 64)):
        row, b0 = 32 * t + l % 32, 64 * s + 32 * (l // 32) + 16 * j
        want = Wq[row, b0:b0 + 16] if row < N else np.zeros(16, np.uint8)
        assert np.array_equal(Wt[t, s, j, l], want)


# (M, N, K, G): streaming kernel, small tiles (with the in-workgroup K split),
# 128 x 256 tiles, ping-pong, ragged N and K, per-channel and coarse groups
SHAPES = [(8, 520, 1024, 128), (32, 8192, 8192, 128), (2, 300, 8224, 8224), (17, 96, 2048, 512),
          (100, 1000, 2048, 128), (300, 520, 4096, 256), (64, 1024, 1024, 1024), (130, 33, 3072, 3072),
          (2048, 8192, 8192, 128), (1111, 8200, 640, 128), (2048, 4096, 8224, 8224), (4096, 2048, 2048, 256)]


@pytest.mark.parametrize("M,N,K,G", SHAPES)
def test_tiled_gemm_equals_row_major(O, M, N, K, G):
    import torch
    m = pk()
    plan = m.apex4_w4a4_gemm_plan("gemm", M, N, K, G, m.APEX4_DEBUG_W_TILED)
    log(f"tiled gemm M={M} N={N} K={K} G={G}: {plan}")
    r = np.random.default_rng(M * 13 + N * 7 + K + G)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    a, s1, w, s2 = (dev(x) for x in (Aq, sa, Wq, sw))
    wt = m.apex4_tile_weights(w)
    Y = m.apex4_w4a4_gemm(a, s1, w, s2, G)
    Yt = m.apex4_w4a4_gemm_tiled(a, s1, wt, s2, G)
    m0, mr = (0, M) if M <= 64 else (M - 40, 36)
    Yd, P = m.apex4_w4a4_gemm_debug(a, s1, wt, s2, G, m0, mr, flags=m.APEX4_DEBUG_W_TILED)
    torch.cuda.synchronize()
    if plan[0] == "gemv":  # two rows on tiled weights: the dot-product kernel
        assert M == 2
        check_tolerance(host(Yt), O.gemm_rows(Aq, sa, Wq, sw, K, G), f"tiled two rows N={N} K={K} G={G}")
    else:
        assert torch.equal(Yt, Y)
    assert torch.equal(Yd, Yt)
    assert np.array_equal(host(P), O.groupsums(Aq, Wq, K, G, m0, mr))


# split over K (workspace entry): ping-pong and small tiles, per channel
SPLIT = [(256, 8192, 8192, 128), (128, 2048, 8192, 256), (256, 4096, 8192, 8192), (300, 2000, 4096, 128)]


@pytest.mark.parametrize("M,N,K,G", SPLIT)
def test_tiled_split_equals_row_major(O, M, N, K, G):
    import torch
    m = pk()
    kern, S = m.apex4_w4a4_gemm_plan("gemm_ws", M, N, K, G, m.APEX4_DEBUG_W_TILED)
    log(f"tiled split M={M} N={N} K={K} G={G}: {kern} S={S}")
    assert S > 1
    r = np.random.default_rng(M + N + K + G)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    a, s1, w, s2 = (dev(x) for x in (Aq, sa, Wq, sw))
    wt = m.apex4_tile_weights(w)
    ws = torch.empty((m.apex4_w4a4_gemm_workspace_size(M, N, K, G),), dtype=torch.uint8, device="cuda")
    Y = m.apex4_w4a4_gemm_ws(a, s1, w, s2, G, ws)
    Yt = m.apex4_w4a4_gemm_tiled(a, s1, wt, s2, G, workspace=ws)
    Yd, P = m.apex4_w4a4_gemm_debug(a, s1, wt, s2, G, 60, 8, workspace=ws, flags=m.APEX4_DEBUG_W_TILED)
    torch.cuda.synchronize()
    assert torch.equal(Yt, Y) and torch.equal(Yd, Y)
    assert np.array_equal(host(P), O.groupsums(Aq, Wq, K, G, 60, 8))


# one row: the tiled one-row kernel (and its fused quantizer)
ONE_ROW = [(1, 8192, 8192, 128), (1, 28672, 8192, 128), (1, 8192, 28672, 128), (1, 1000, 4096, 256),
           (1, 257, 2048, 1024), (1, 300, 3072, 3072), (1, 33, 8224, 8224), (1, 520, 8192, 512), (1, 100, 122880, 128)]


@pytest.mark.parametrize("M,N,K,G", ONE_ROW)
def test_tiled_one_row(O, M, N, K, G):
    import torch
    m = pk()
    log(f"tiled one row N={N} K={K} G={G}: gemm {m.apex4_w4a4_gemm_plan('gemm', M, N, K, G, m.APEX4_DEBUG_W_TILED)}, "
        f"linear {m.apex4_w4a4_gemm_plan('linear', M, N, K, G, m.APEX4_DEBUG_W_TILED)}")
    w = wl.weights(wl.rng_for("decode", 7, N + K), N, K)
    x = wl.activations(wl.rng_for("decode", 8, K + G), M, K)
    Wq_d, sw_d = m.apex4_quantize_act(dev(w), G)
    Wt = m.apex4_tile_weights(Wq_d)
    Aq_d, sa_d = m.apex4_quantize_act(dev(x), G)
    Y = m.apex4_w4a4_gemm_tiled(Aq_d, sa_d, Wt, sw_d, G)
    Aw = torch.full((M, K // 2), 0xAB, dtype=torch.uint8, device="cuda")
    saw = torch.full((M, K // G), float("nan"), dtype=torch.float16, device="cuda")
    Yl = m.apex4_w4a4_linear_tiled(dev(x), Wt, sw_d, G, A_q_work=Aw, s_a_work=saw)
    Yd, P = m.apex4_w4a4_gemm_debug(Aq_d, sa_d, Wt, sw_d, G, flags=m.APEX4_DEBUG_W_TILED)
    Yld, _, _, Pl = m.apex4_w4a4_linear_debug(dev(x), Wt, sw_d, G, flags=m.APEX4_DEBUG_W_TILED)
    torch.cuda.synchronize()
    assert torch.equal(Aw, Aq_d) and torch.equal(saw.view(torch.int16), sa_d.view(torch.int16))
    assert torch.equal(Yl, Y) and torch.equal(Yd, Y) and torch.equal(Yld, Y)
    Wq_o, sw_o = O.quantize(w, G)
    Aq_o, sa_o = O.quantize(x, G)
    assert np.array_equal(host(Wq_d), Wq_o) and np.array_equal(host(Aq_d), Aq_o)
    P_o = O.groupsums(Aq_o, Wq_o, K, G)
    assert np.array_equal(host(P), P_o) and np.array_equal(host(Pl), P_o)
    check_tolerance(host(Y), O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G), f"tiled one row N={N} K={K} G={G}")


# two rows: the two-row form of the tiled dot-product kernel (ragged N, K past
# 64 KB of codes per row, G > 128 with sub-group partials, per channel)
TWO_ROWS = [(2, 8192, 8192, 128), (2, 28672, 8192, 128), (2, 10240, 8192, 128), (2, 8192, 28672, 128),
            (2, 1000, 4096, 256), (2, 257, 2048, 1024), (2, 300, 3072, 3072), (2, 33, 8224, 8224),
            (2, 520, 8192, 512), (2, 100, 57344, 128)]


@pytest.mark.parametrize("M,N,K,G", TWO_ROWS)
def test_tiled_two_rows(O, M, N, K, G):
    import torch
    m = pk()
    T = m.APEX4_DEBUG_W_TILED
    plans = (m.apex4_w4a4_gemm_plan("gemm", M, N, K, G, T), m.apex4_w4a4_gemm_plan("linear", M, N, K, G, T),
             m.apex4_w4a4_gemm_plan("gemm", M, N, K, G))
    log(f"tiled two rows N={N} K={K} G={G}: gemm {plans[0]}, linear {plans[1]}, row-major {plans[2]}")
    assert plans[0] == ("gemv", 1) and plans[1] == ("gemv", 1) and plans[2] == ("decode", 1)
    w = wl.weights(wl.rng_for("decode", 17, N + K), N, K)
    x = wl.activations(wl.rng_for("decode", 18, K + G), M, K)
    Wq_d, sw_d = m.apex4_quantize_act(dev(w), G)
    Wt = m.apex4_tile_weights(Wq_d)
    Aq_d, sa_d = m.apex4_quantize_act(dev(x), G)
    Y = m.apex4_w4a4_gemm_tiled(Aq_d, sa_d, Wt, sw_d, G)
    Aw = torch.full((M, K // 2), 0xAB, dtype=torch.uint8, device="cuda")
    saw = torch.full((M, K // G), float("nan"), dtype=torch.float16, device="cuda")
    Yl = m.apex4_w4a4_linear_tiled(dev(x), Wt, sw_d, G, A_q_work=Aw, s_a_work=saw)
    dumps = [m.apex4_w4a4_gemm_debug(Aq_d, sa_d, Wt, sw_d, G, m0, mr, flags=T) for m0, mr in ((0, 2), (1, 1), (0, 1))]
    Yld, _, _, Pl = m.apex4_w4a4_linear_debug(dev(x), Wt, sw_d, G, flags=T)
    torch.cuda.synchronize()
    assert torch.equal(Aw, Aq_d) and torch.equal(saw.view(torch.int16), sa_d.view(torch.int16))
    assert torch.equal(Yl, Y) and torch.equal(Yld, Y) and all(torch.equal(Yd, Y) for Yd, _ in dumps)
    Wq_o, sw_o = O.quantize(w, G)
    Aq_o, sa_o = O.quantize(x, G)
    assert np.array_equal(host(Wq_d), Wq_o) and np.array_equal(host(Aq_d), Aq_o)
    P_o = O.groupsums(Aq_o, Wq_o, K, G)
    assert np.array_equal(host(Pl), P_o)
    for (m0, mr), (_, P) in zip(((0, 2), (1, 1), (0, 1)), dumps):
        assert np.array_equal(host(P), P_o[m0:m0 + mr]), (m0, mr)
    check_tolerance(host(Y), O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G), f"tiled two rows N={N} K={K} G={G}")


@pytest.mark.parametrize("M", [5, 32, 300])
def test_tiled_linear(O, M):
    import torch
    m = pk()
    N, K, G = 1000, 4096, 128
    w = wl.weights(wl.rng_for("decode", 9, M), N, K)
    x = wl.activations(wl.rng_for("decode", 10, M), M, K)
    Wq_d, sw_d = m.apex4_quantize_act(dev(w), G)
    Wt = m.apex4_tile_weights(Wq_d)
    Yl = m.apex4_w4a4_linear_tiled(dev(x), Wt, sw_d, G)
    Y = m.apex4_w4a4_linear(dev(x), Wq_d, sw_d, G)
    torch.cuda.synchronize()
    assert torch.equal(Yl, Y)
    Wq_o, sw_o = O.quantize(w, G)
    Aq_o, sa_o = O.quantize(x, G)
    check_tolerance(host(Yl), O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G), f"tiled linear M={M}")


def test_tiled_extreme_codes(O):
    """All codes -8 (7 on even weight rows) through the tiled one-row, streaming and tile kernels."""
    import torch
    m = pk()
    N, K = 72, 4096
    for M, G in ((1, 128), (8, 256), (100, 128), (64, 4096)):
        Aq = np.full((M, K // 2), 0x88, np.uint8)
        Wq = np.full((N, K // 2), 0x88, np.uint8)
        Wq[::2] = 0x77
        s_a = np.full((M, K // G), 2.0 ** -7, np.float16)
        s_w = np.full((N, K // G), 2.0 ** -7, np.float16)
        a, s1, w, s2 = (dev(v) for v in (Aq, s_a, Wq, s_w))
        Yd, P = m.apex4_w4a4_gemm_debug(a, s1, m.apex4_tile_weights(w), s2, G, flags=m.APEX4_DEBUG_W_TILED)
        torch.cuda.synchronize()
        assert np.array_equal(host(P), O.groupsums(Aq, Wq, K, G))
        check_tolerance(host(Yd), O.gemm_rows(Aq, s_a, Wq, s_w, K, G), f"tiled extreme M={M} G={G}")
