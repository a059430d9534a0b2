"""GPU parity of the W4A4 group GEMM (APEX4 Sec. 3.2.1, Eq. group_decomposition).

  * integer group sums from the GEMM kernel's dump epilogue are bit-identical to
    the oracle's int64 sums;
  * the binary16 output is within |Y - y| <= 2e-3 |y| + 1e-2 RMS_row(y) of the
    oracle's binary64 y;
  * workloads: tiny (M=64, N=K=1024) in full, the paper shape (M=2048,
    N=K=8192, G=128) on sampled rows, the Llama-2-70B linears, the granularity
    sweep and the decode path, plus ragged and degenerate shapes, and operands
    of the largest size the ABI accepts (just under 4 GiB).

For the float workloads both sides quantize the same binary16 inputs
independently (oracle quantizer on the host, HIP quantizer on the device).
"""
import numpy as np
import pytest

from parity import check_tolerance, dev, host, log, sample_rows
from paper_2606_08761_amd import workloads as wl

pytestmark = pytest.mark.gpu


def pk():
    import paper_2606_08761_amd as m
    return m


def run_gemm(Aq, sa, Wq, sw, G):
    return host(pk().apex4_w4a4_gemm(dev(Aq), dev(sa), dev(Wq), dev(sw), G))


def run_groupsums(Aq, Wq, G, m0=0, mr=None):
    return host(pk().apex4_w4a4_gemm_groupsums(dev(Aq), dev(Wq), G, m0, mr))


def test_tiny_workload_full(O):
    M, N, K, G = 64, 1024, 1024, 128
    log("tiny workload")
    Aq, sa, Wq, sw = wl.codes_workload("tiny", M, N, K, G)
    P = run_groupsums(Aq, Wq, G)
    assert np.array_equal(P.astype(np.int64), O.groupsums(Aq, Wq, K, G))
    check_tolerance(run_gemm(Aq, sa, Wq, sw, G), O.gemm_rows(Aq, sa, Wq, sw, K, G), "tiny")


# Ragged shapes with at least one 128 x 256 tile per CU: G = 128 runs the
# ping-pong kernel there (partial M and N tiles, odd N, an odd stage count).
BIG_RAGGED = [(1111, 8200, 640, 128), (1500, 8195, 1152, 128), (2050, 4100, 4096, 128)]


@pytest.mark.parametrize("M,N,K,G", BIG_RAGGED)
def test_big_ragged_shapes(O, M, N, K, G):
    log(f"big ragged M={M} N={N} K={K} G={G}")
    r = np.random.default_rng(M * 7919 + N * 31 + K + G + 1)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    check_tolerance(run_gemm(Aq, sa, Wq, sw, G), O.gemm_rows(Aq, sa, Wq, sw, K, G), f"big ragged {M}x{N}x{K} G{G}")


RAGGED = [
    (1, 128, 128, 128), (8, 200, 256, 128), (33, 1024, 1024, 256), (129, 136, 512, 512),
    (2, 64, 1024, 1024), (300, 260, 384, 128), (64, 1024, 1024, 1024), (17, 8, 256, 256),
    (255, 257, 768, 256), (128, 128, 2048, 512), (1, 1, 128, 128), (130, 33, 3072, 3072),
    (64, 300, 1024, 32), (130, 520, 1536, 64), (3, 40, 512, 32), (200, 264, 4096, 1024),
    (400, 1000, 2048, 32), (9, 96, 2048, 1024),
]


@pytest.mark.parametrize("M,N,K,G", RAGGED)
def test_ragged_shapes(O, M, N, K, G):
    log(f"ragged M={M} N={N} K={K} G={G}")
    r = np.random.default_rng(M * 7919 + N * 31 + K + G)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    P = run_groupsums(Aq, Wq, G)
    assert np.array_equal(P.astype(np.int64), O.groupsums(Aq, Wq, K, G))
    check_tolerance(run_gemm(Aq, sa, Wq, sw, G), O.gemm_rows(Aq, sa, Wq, sw, K, G), f"ragged {M}x{N}x{K} G{G}")


@pytest.mark.parametrize("G", [32, 64, 128, 256, 512, 1024])
def test_extreme_codes(O, G):
    """Every code -8: P = 64 G per group, the largest magnitude the int32 path sees."""
    M, N, K = 40, 72, 1024
    Aq = np.full((M, K // 2), 0x88, np.uint8)
    Wq = np.full((N, K // 2), 0x88, np.uint8)
    Wq[::2] = 0x77                                           # and 7 * -8 = -56 on even rows
    P = run_groupsums(Aq, Wq, G)
    assert np.array_equal(P.astype(np.int64), O.groupsums(Aq, Wq, K, G))
    # scales 2^-6 keep y = 64 K 2^-12 inside binary16 (unit scales would give 65536 -> inf)
    s_a = np.full((M, K // G), 2.0 ** -6, np.float16)
    s_w = np.full((N, K // G), 2.0 ** -6, np.float16)
    check_tolerance(run_gemm(Aq, s_a, Wq, s_w, G), O.gemm_rows(Aq, s_a, Wq, s_w, K, G), "extreme")


def test_paper_shape_sampled(O):
    """M=2048, N=K=8192, G=128 in the launch configuration the benchmark times."""
    M, N, K, G = 2048, 8192, 8192, 128
    log("paper shape: generate")
    Aq, sa, Wq, sw = wl.codes_workload("paper", M, N, K, G)
    Y = run_gemm(Aq, sa, Wq, sw, G)
    rows = sample_rows(M, seed=1)
    log(f"paper shape: oracle rows {rows.tolist()}")
    check_tolerance(Y[rows], O.gemm_rows(Aq, sa, Wq, sw, K, G, rows), "paper shape")
    for m0, mr in ((0, 4), (126, 4), (2044, 4)):
        P = run_groupsums(Aq, Wq, G, m0, mr)
        assert np.array_equal(P.astype(np.int64), O.groupsums(Aq, Wq, K, G, m0, mr)), (m0, mr)


class Weights:
    """A binary16 weight matrix quantized on both sides (once)."""

    def __init__(self, O, w, G):
        m = pk()
        self.N, self.K, self.G = w.shape[0], w.shape[1], G
        self.Wq_d, self.sw_d = m.apex4_quantize_act(dev(w), G)
        self.Wq_o, self.sw_o = O.quantize(w, G)
        wrows = sample_rows(self.N, seed=3)
        assert np.array_equal(host(self.Wq_d)[wrows], self.Wq_o[wrows])
        assert np.array_equal(host(self.sw_d)[wrows].view(np.uint16), self.sw_o[wrows].view(np.uint16))


def _float_case(O, name, W, x, rows):
    """Quantize x on both sides, compare codes on the sampled rows, then Y."""
    import torch
    m = pk()
    G, K = W.G, W.K
    Aq_d, sa_d = m.apex4_quantize_act(dev(x), G)
    Y = host(m.apex4_w4a4_gemm(Aq_d, sa_d, W.Wq_d, W.sw_d, G))
    torch.cuda.synchronize()
    Aq_o, sa_o = O.quantize(x[rows], G)
    assert np.array_equal(host(Aq_d)[rows], Aq_o), name
    assert np.array_equal(host(sa_d)[rows].view(np.uint16), sa_o.view(np.uint16)), name
    y = O.gemm_rows(Aq_o, sa_o, W.Wq_o, W.sw_o, K, G)
    check_tolerance(Y[rows], y, name)
    return Y


@pytest.mark.parametrize("linear", list(wl.LLAMA70B_LINEARS))
def test_llama70b_linears(O, linear):
    N, K = wl.LLAMA70B_LINEARS[linear]
    G = 128
    log(f"llama70b {linear}: generate weights {N}x{K}")
    W = Weights(O, wl.weights(wl.rng_for("llama70b", 10 + list(wl.LLAMA70B_LINEARS).index(linear)), N, K), G)
    for M in (16, 256, 4096):
        log(f"llama70b {linear} M={M}")
        x = wl.activations(wl.rng_for("llama70b", 20, M * 100 + K // 1024), M, K)
        rows = sample_rows(M, seed=M, n_random=4) if M > 16 else np.arange(M)
        _float_case(O, f"{linear} M={M}", W, x, rows)


# The paper's mixed configuration (Sec. 3.2.2) on Llama-2-70B shapes: the value
# projection (N=1024) and the down projection (K=28672, 896 groups) at G=32, the
# query+key projection (N=9216) per channel; decode and batched rows.
MIXED = [("v", 1024, 8192, 32), ("down", 8192, 28672, 32), ("qk", 9216, 8192, 8192)]


@pytest.mark.parametrize("name,N,K,G", MIXED)
def test_mixed_granularity_linears(O, name, N, K, G):
    log(f"mixed {name}: generate weights {N}x{K} G={G}")
    W = Weights(O, wl.weights(wl.rng_for("llama70b", 30 + K // 1024 + N // 1024), N, K), G)
    for M in (16, 256):
        log(f"mixed {name} M={M}")
        x = wl.activations(wl.rng_for("llama70b", 31, M * 100 + K // 1024), M, K)
        rows = sample_rows(M, seed=M + 7, n_random=4) if M > 16 else np.arange(M)
        _float_case(O, f"mixed {name} M={M}", W, x, rows)


@pytest.mark.parametrize("G", [128, 256, 512, 8192])
def test_granularity_sweep(O, G):
    M, N, K = 4096, 8192, 8192
    log(f"gsweep G={G}")
    W = Weights(O, wl.weights(wl.rng_for("gsweep", 2), N, K), G)
    x = wl.activations(wl.rng_for("gsweep", 1, G), M, K)
    _float_case(O, f"gsweep G={G}", W, x, sample_rows(M, seed=G, n_random=4))


@pytest.mark.parametrize("N,K", [(8192, 8192), (28672, 8192)])
def test_decode_linear(O, N, K):
    """The quantize + GEMM linear entry point at decode sizes, every row checked."""
    import torch
    G = 128
    m = pk()
    w = wl.weights(wl.rng_for("decode", 2, N), N, K)
    Wq_o, sw_o = O.quantize(w, G)
    Wq_d, sw_d = m.apex4_quantize_act(dev(w), G)
    for M in (1, 8, 32):
        log(f"decode N={N} K={K} M={M}")
        x = wl.activations(wl.rng_for("decode", 1, M * 1000 + N // 1024), M, K)
        Y = m.apex4_w4a4_linear(dev(x), Wq_d, sw_d, G)
        torch.cuda.synchronize()
        Aq_o, sa_o = O.quantize(x, G)
        check_tolerance(host(Y), O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G), f"decode M={M}")
        # the linear entry point equals quantize-then-GEMM bit for bit
        Aq_d, sa_d = m.apex4_quantize_act(dev(x), G)
        Y2 = m.apex4_w4a4_gemm(Aq_d, sa_d, Wq_d, sw_d, G)
        assert torch.equal(Y, Y2)


# (M, N, K, G) of the linear entry point at one row.  The fused quantize + GEMM
# kernel (G in {32, 64, 128, 256, 512}, G < K, when its redundant prologue work
# is small) takes: Llama-2-70B o_proj and v_proj sizes, ragged N, a partial
# last 1 KB chunk (K = 1536), every fused G, and K = 122880, the largest whose
# codes and scales fit the kernel's 64 KiB of LDS.  The rest take the two
# kernels: larger N x K (gate/up, down), K = 131072 (does not fit), two rows,
# G = K and G = 1024.  Either way the result must equal quantize-then-GEMM.
FUSED = [(1, 8192, 8192, 128), (1, 1024, 8192, 128), (1, 1000, 4096, 256), (1, 520, 8192, 512),
         (1, 33, 1024, 512), (1, 96, 1536, 128), (1, 1024, 8192, 32), (1, 520, 4096, 64), (1, 200, 122880, 128),
         (1, 28672, 8192, 128), (1, 8192, 28672, 128), (1, 200, 131072, 128), (2, 200, 4096, 128),
         (1, 64, 4096, 4096), (1, 72, 8192, 1024)]


@pytest.mark.parametrize("M,N,K,G", FUSED)
def test_fused_linear(O, M, N, K, G):
    """The linear entry point's one-kernel path: Y and the work buffers equal
    apex4_quantize_act followed by apex4_w4a4_gemm bit for bit, and Y is within
    tolerance of the oracle on every row."""
    import torch
    m = pk()
    log(f"fused linear M={M} N={N} K={K} G={G}")
    w = wl.weights(wl.rng_for("decode", 5, N * 7 + K), N, K)
    x = wl.activations(wl.rng_for("decode", 6, M * 1000 + K // 128 + G), M, K)
    Wq_d, sw_d = m.apex4_quantize_act(dev(w), G)
    Aq_w = torch.full((M, K // 2), 0xAB, dtype=torch.uint8, device="cuda")
    sa_w = torch.full((M, K // G), float("nan"), dtype=torch.float16, device="cuda")
    Y = m.apex4_w4a4_linear(dev(x), Wq_d, sw_d, G, A_q_work=Aq_w, s_a_work=sa_w)
    Aq_d, sa_d = m.apex4_quantize_act(dev(x), G)
    Y2 = m.apex4_w4a4_gemm(Aq_d, sa_d, Wq_d, sw_d, G)
    torch.cuda.synchronize()
    assert torch.equal(Aq_w, Aq_d)
    assert torch.equal(sa_w.view(torch.int16), sa_d.view(torch.int16))
    assert torch.equal(Y, Y2)
    Wq_o, sw_o = O.quantize(w, G)
    Aq_o, sa_o = O.quantize(x, G)
    check_tolerance(host(Y), O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G), f"fused M={M} N={N} K={K} G={G}")


DECODE = [
    (1, 96, 4224, 128), (5, 40, 2560, 512), (32, 300, 1536, 1536), (16, 64, 28672, 256),
    (3, 1000, 1152, 128), (31, 33, 640, 128), (32, 8192, 8192, 512), (8, 520, 8192, 1024),
    (4, 300, 2048, 64), (32, 1024, 1024, 32),
    # G = 32 and 64 on the streaming kernel: the mixed configuration's value
    # (N=1024, K=8192) and down (K=28672) projections at decode batch sizes
    (16, 1024, 8192, 32), (16, 2048, 28672, 32), (1, 520, 4096, 64), (9, 96, 8192, 32), (32, 64, 2048, 64),
    # one row (the dot-product kernel): every G, G = K not a power of two,
    # partial last chunks (K/2 not a multiple of 1 KB), N below one wave's share
    (1, 1000, 8192, 32), (1, 257, 2048, 1024), (1, 300, 3072, 3072), (1, 8192, 28672, 128),
    (1, 3, 640, 128), (1, 4097, 8192, 256), (1, 100, 122880, 512),
]


@pytest.mark.parametrize("M,N,K,G", DECODE)
def test_decode_kernel_shapes(O, M, N, K, G):
    """Up to 32 rows run on the weight-streaming kernel (K split over 8 waves),
    one row on the dot-product kernel."""
    log(f"decode kernel M={M} N={N} K={K} G={G}")
    r = np.random.default_rng(M * 104729 + N * 13 + K + G)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    check_tolerance(run_gemm(Aq, sa, Wq, sw, G), O.gemm_rows(Aq, sa, Wq, sw, K, G), f"decode {M}x{N}x{K} G{G}")


@pytest.mark.parametrize("G", [32, 64, 128, 512])
def test_decode_extreme_codes(O, G):
    M, N, K = 8, 72, 2048
    Aq = np.full((M, K // 2), 0x88, np.uint8)
    Wq = np.full((N, K // 2), 0x88, np.uint8)
    Wq[::2] = 0x77
    s_a = np.full((M, K // G), 2.0 ** -7, np.float16)
    s_w = np.full((N, K // G), 2.0 ** -7, np.float16)
    check_tolerance(run_gemm(Aq, s_a, Wq, s_w, G), O.gemm_rows(Aq, s_a, Wq, s_w, K, G), "decode extreme")


def test_decode_repeatable():
    import torch
    m = pk()
    M, N, K, G = 16, 520, 3072, 128
    Aq, sa, Wq, sw = wl.codes_workload("tiny", M, N, K, G)
    a, s1, w, s2 = dev(Aq), dev(sa), dev(Wq), dev(sw)
    Y1 = m.apex4_w4a4_gemm(a, s1, w, s2, G)
    for _ in range(5):
        assert torch.equal(m.apex4_w4a4_gemm(a, s1, w, s2, G), Y1)


@pytest.mark.parametrize("G", [32, 64, 1024])
def test_fine_and_coarse_groups_float_workload(O, G):
    """The paper's other granularities (Sec. 3.2.2): activations and weights quantized
    on the device with G, every output element checked; exact group sums on a row window."""
    M, N, K = 256, 1024, 4096
    log(f"granularity G={G} M={M} N={N} K={K}")
    x, w = wl.float_workload("gsweep", M, N, K)
    m = pk()
    Aq_d, sa_d = m.apex4_quantize_act(dev(x), G)
    Wq_d, sw_d = m.apex4_quantize_act(dev(w), G)
    Aq_o, sa_o = O.quantize(x, G)
    Wq_o, sw_o = O.quantize(w, G)
    assert np.array_equal(host(Aq_d), Aq_o) and np.array_equal(host(Wq_d), Wq_o)
    check_tolerance(host(m.apex4_w4a4_gemm(Aq_d, sa_d, Wq_d, sw_d, G)), O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G),
                    f"G={G}")
    P = host(m.apex4_w4a4_gemm_groupsums(Aq_d, Wq_d, G, 100, 40))
    assert np.array_equal(P.astype(np.int64), O.groupsums(Aq_o[100:140], Wq_o, K, G))


def test_repeatable_and_degenerate():
    import torch
    m = pk()
    M, N, K, G = 300, 520, 1024, 128
    Aq, sa, Wq, sw = wl.codes_workload("tiny", M, N, K, G)
    a, s1, w, s2 = dev(Aq), dev(sa), dev(Wq), dev(sw)
    Y1 = m.apex4_w4a4_gemm(a, s1, w, s2, G)
    for _ in range(5):
        assert torch.equal(m.apex4_w4a4_gemm(a, s1, w, s2, G), Y1)
    P1 = m.apex4_w4a4_gemm_groupsums(a, w, G)
    assert torch.equal(m.apex4_w4a4_gemm_groupsums(a, w, G), P1)
    # M == 0 and an empty row window are successful no-ops
    m.apex4_w4a4_gemm(a[:0], s1[:0], w, s2, G)
    m.apex4_w4a4_gemm_groupsums(a, w, G, 5, 0)
    torch.cuda.synchronize()


def _untile(Wt, N, K):
    """Row-major packed codes back from the tiled layout (its definition, inverted)."""
    T, S = -(-N // 32), -(-K // 128)
    v = Wt.reshape(T, S, 2, 2, 32, 16)             # [t][s][j][h][c][b], lane = 32 h + c
    rows = v.transpose(0, 4, 1, 3, 2, 5).reshape(T * 32, S * 64)
    return rows[:N, :K // 2]


def test_w4a4_linear_module(O):
    """The drop-in layer: offline weight quantization (tiled layout by default,
    row-major on request) + per-call activation quantization and GEMM, batched
    leading dimensions, work buffers reused per (rows, stream)."""
    import torch
    m = pk()
    N, K, G = 1024, 2048, 128
    x, w = wl.float_workload("tiny", 64, N, K)
    Wq_o, sw_o = O.quantize(w, G)
    lin = m.W4A4Linear(dev(w), G)
    lin_r = m.W4A4Linear(dev(w), G, layout="rows")
    assert lin.tiled and lin.W_q is None and not lin_r.tiled
    assert np.array_equal(_untile(host(lin.W_t), N, K), Wq_o)
    assert np.array_equal(host(lin_r.W_q), Wq_o)
    stream = torch.cuda.current_stream()
    # same shape twice (buffers reused), then others; 64 rows take the split-K
    # GEMM with the layer's own workspace
    for rows in (24, 24, 7, 64):
        xb = x[:rows]
        y = lin(dev(xb).reshape(1, rows, K))
        yr = lin_r(dev(xb).reshape(1, rows, K))
        torch.cuda.synchronize()
        assert y.shape == (1, rows, N)
        assert torch.equal(y, yr)                  # rows > 1: the same bits from either layout
        assert (lin._work[(rows, stream.cuda_stream)][2] is not None) == (rows == 64)
        Aq_o, sa_o = O.quantize(xb, G)
        check_tolerance(host(y)[0], O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G), f"module rows={rows}")
    assert len(lin._work) == 3
    # one row (the one-row kernels) through both layouts
    y1, y1r = host(lin(dev(x[:1]))), host(lin_r(dev(x[:1])))
    Aq_o, sa_o = O.quantize(x[:1], G)
    for yy in (y1, y1r):
        check_tolerance(yy, O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G), "module one row")
    # per-channel weights through the same layer
    lin_c = m.W4A4Linear(dev(w), 0)
    assert lin_c.tiled
    Wq_c, sw_c = O.quantize(w, K)
    Aq_c, sa_c = O.quantize(x[:24], K)
    check_tolerance(host(lin_c(dev(x[:24]))), O.gemm_rows(Aq_c, sa_c, Wq_c, sw_c, K, K), "module per-channel")
    # G < 128 keeps row-major weights
    lin_32 = m.W4A4Linear(dev(w), 32)
    assert not lin_32.tiled
    with pytest.raises(ValueError):
        m.W4A4Linear(dev(w), 32, layout="tiled")
    torch.cuda.synchronize()


def test_w4a4_linear_module_streams(O):
    """Forwards with the same row count on two streams use separate work
    buffers: both results are right although the streams overlap."""
    import torch
    m = pk()
    N, K, G, rows = 2048, 4096, 128, 64
    x, w = wl.float_workload("tiny", 2 * rows, N, K)
    lin = m.W4A4Linear(dev(w), G)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    xa, xb = dev(x[:rows]), dev(x[rows:])
    torch.cuda.synchronize()
    with torch.cuda.stream(s1):
        ya = lin(xa)
    with torch.cuda.stream(s2):
        yb = lin(xb)
    torch.cuda.synchronize()
    assert len(lin._work) == 2
    Wq_o, sw_o = O.quantize(w, G)
    for xx, yy in ((x[:rows], ya), (x[rows:], yb)):
        Aq_o, sa_o = O.quantize(xx, G)
        check_tolerance(host(yy), O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G), "module two streams")


def test_w4a4_linear_module_graph(O):
    """The drop-in layer captured in a graph, as a serving loop would: one row
    (the fused kernel), 16 rows (the few-row kernel's stream-K form) and 64
    rows (split over K), each with the layer's own work buffers.  Three
    replays with eager calls of the same layer in between each give the eager
    bits, and those are within the oracle's tolerance."""
    import torch
    m = pk()
    N, K, G = 1024, 8192, 32
    x, w = wl.float_workload("tiny", 64, N, K)
    lin = m.W4A4Linear(dev(w), G)
    xs = {r: dev(x[:r]) for r in (1, 16, 64)}
    plans = {r: m.apex4_w4a4_gemm_plan("gemm_ws", r, N, K, G) for r in (16, 64)}
    log(f"module graph: plans {plans}")
    assert plans[16] == ("decode_split", 1) and plans[64][1] > 1
    eager = {r: lin(xs[r]) for r in xs}
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        outs = {r: lin(xs[r]) for r in xs}
    torch.cuda.synchronize()
    for i in range(3):
        for yy in outs.values():
            yy.fill_(float("nan"))
        again = {r: lin(xs[r]) for r in xs}   # eager work on the device between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for r in xs:
            assert torch.equal(outs[r], eager[r]) and torch.equal(again[r], eager[r]), (i, r)
    Wq_o, sw_o = O.quantize(w, G)
    for r in xs:
        Aq_o, sa_o = O.quantize(x[:r], G)
        check_tolerance(host(eager[r]), O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G), f"module graph rows={r}")


def test_weights_just_under_4gib(O):
    """The largest weight operand the ABI accepts: N K/2 = 4,294,950,912 bytes,
    16 KiB under 2^32 (the kernels address operand rows with 32-bit byte
    offsets).  One row (dot-product kernel), 8 rows (decode kernel) and 40
    rows (tile kernel), checked on sampled output columns that include the
    last rows of W."""
    import torch
    m = pk()
    N, K, G = 262143, 32768, 128
    assert N * (K // 2) < 2 ** 32 and (N + 1) * (K // 2) >= 2 ** 32
    log("4 GiB weights: generate")
    r = np.random.default_rng(4096)
    Wq = wl.random_codes(r, N, K)
    sw = wl.random_scales(r, N, K // G)
    Wq_d, sw_d = dev(Wq), dev(sw)
    cols = np.unique(np.concatenate([np.arange(8), np.arange(N - 8, N), r.integers(0, N, size=24)]))
    Wq_s, sw_s = Wq[cols], sw[cols]
    del Wq
    for M in (1, 8, 40):
        log(f"4 GiB weights: M={M}")
        Aq, sa = wl.random_codes(r, M, K), wl.random_scales(r, M, K // G)
        Y = host(m.apex4_w4a4_gemm(dev(Aq), dev(sa), Wq_d, sw_d, G))
        assert Y.shape == (M, N)
        check_tolerance(Y[:, cols], O.gemm_rows(Aq, sa, Wq_s, sw_s, K, G), f"4 GiB weights M={M}")
    del Wq_d, sw_d
    torch.cuda.empty_cache()


def test_activations_just_under_4gib(O):
    """The largest activation operand: M K/2 = 4,294,950,912 bytes (tile kernel,
    32-bit row offsets), checked on sampled rows that include the last ones."""
    import torch
    m = pk()
    M, N, K, G = 262143, 40, 32768, 128
    log("4 GiB activations: generate")
    r = np.random.default_rng(4097)
    Aq = wl.random_codes(r, M, K)
    sa = wl.random_scales(r, M, K // G)
    Wq, sw = wl.random_codes(r, N, K), wl.random_scales(r, N, K // G)
    Y = host(m.apex4_w4a4_gemm(dev(Aq), dev(sa), dev(Wq), dev(sw), G))
    rows = np.unique(np.concatenate([np.arange(4), np.arange(M - 130, M), r.integers(0, M, size=16)]))
    check_tolerance(Y[rows], O.gemm_rows(Aq, sa, Wq, sw, K, G, rows), "4 GiB activations")
    torch.cuda.empty_cache()
