"""GPU parity of the MX numerics variant (power-of-two group scales in the
block-scaled FP6 MFMA), against oracle/mx.py.

  * apex4_quantize_mx: FP6 codes and E8M0 bytes bit-identical to the oracle's
    (codes re-encoded on the host with oracle.fp6), on the realistic
    activation distribution and on edge groups (zeros, subnormals, fp16 max,
    exact 7 * 2^e boundaries, ties);
  * apex4_w4a4_gemm_mx: within |Y - y| <= 2e-3 |y| + 1e-2 RMS_row(y) of the
    oracle's binary64 y, fed with oracle-quantized operands (independent of the
    GPU quantizer) and end to end from fp16 inputs;
  * group sizes 32 .. 1024, ragged and degenerate shapes, the M=2048 N=K=8192
    shape on sampled rows.
"""
import numpy as np
import pytest

from oracle import fp6 as ofp6
from oracle import mx as omx
from parity import check_tolerance, dev, host, log, sample_rows
from paper_2606_08761_amd import workloads as wl

pytestmark = pytest.mark.gpu


def pk():
    import paper_2606_08761_amd as m
    return m


def quantize_both(x, G):
    Q6, e = pk().apex4_quantize_mx(dev(x), G)
    codes_o, e_o = omx.quantize_mx(x, G)
    return host(Q6), host(e), codes_o, e_o


@pytest.mark.parametrize("M,K,G", [(64, 1024, 128), (37, 384, 32), (5, 2048, 64), (300, 1024, 256),
                                   (8, 4096, 512), (3, 2048, 1024), (129, 8192, 128)])
def test_quantizer_bit_exact(M, K, G):
    log(f"mx quantize M={M} K={K} G={G}")
    x = wl.activations(wl.rng_for("tiny", 50, M * 100000 + K + G), M, K)
    Q6, e, codes_o, e_o = quantize_both(x, G)
    assert np.array_equal(e, e_o)
    assert np.array_equal(Q6, ofp6.pack_fp6(codes_o))


def test_quantizer_edge_groups():
    K, G = 256, 32
    rows = []
    z = np.zeros(K, np.float16)
    rows.append(z.copy())                                             # all zero
    r = z.copy(); r[:32] = np.float16(2.0 ** -24); rows.append(r)     # smallest subnormal
    r = z.copy(); r[3] = np.float16(65504.0); r[4] = np.float16(-65504.0); rows.append(r)   # fp16 max
    r = z.copy(); r[0] = 7.0; r[1] = 3.5; r[2] = -2.5; r[3] = 0.5; rows.append(r)           # E = 0 boundary, ties
    r = z.copy(); r[0] = np.float16(np.nextafter(np.float16(7.0), np.float16(8.0))); r[1] = 3.5; rows.append(r)
    r = z.copy(); r[32:64] = np.linspace(-1e-3, 1e-3, 32).astype(np.float16); rows.append(r)
    r = z.copy(); r[::2] = -0.0; r[1] = -6.0; rows.append(r)
    x = np.stack(rows).astype(np.float16)
    Q6, e, codes_o, e_o = quantize_both(x, G)
    assert np.array_equal(e, e_o)
    assert np.array_equal(Q6, ofp6.pack_fp6(codes_o))


def gemm_from_oracle_operands(Aq, ea, Wq, ew, G):
    m = pk()
    return host(m.apex4_w4a4_gemm_mx(dev(ofp6.pack_fp6(Aq)), dev(ea), dev(ofp6.pack_fp6(Wq)), dev(ew), G))


@pytest.mark.parametrize("M,N,K,G", [(64, 1024, 1024, 128), (1, 1, 128, 128), (8, 200, 256, 32), (300, 260, 384, 64),
                                     (129, 136, 512, 256), (33, 1000, 1024, 1024), (1111, 8200, 640, 128),
                                     (255, 257, 768, 32), (2050, 4100, 2048, 512)])
def test_gemm_oracle_operands(O, M, N, K, G):
    log(f"mx gemm M={M} N={N} K={K} G={G}")
    r = np.random.default_rng(M * 31 + N * 7 + K + G)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    ea = (127 + r.integers(-6, 3, size=(M, K // G))).astype(np.uint8)
    ew = (127 + r.integers(-6, 3, size=(N, K // G))).astype(np.uint8)
    Y = gemm_from_oracle_operands(Aq, ea, Wq, ew, G)
    rows = sample_rows(M, seed=M) if M > 64 else np.arange(M)
    check_tolerance(Y[rows], omx.gemm_mx_f64(Aq, ea, Wq, ew, K, G, rows), f"mx {M}x{N}x{K} G{G}")


@pytest.mark.parametrize("G", [32, 128, 1024])
def test_end_to_end_from_fp16(G):
    """GPU quantizer + GPU GEMM against the oracle's quantize + GEMM of the same fp16 inputs."""
    M, N, K = 256, 1024, 2048
    log(f"mx end to end G={G}")
    x, w = wl.float_workload("tiny", M, N, K)
    m = pk()
    A6, ea = m.apex4_quantize_mx(dev(x), G)
    W6, ew = m.apex4_quantize_mx(dev(w), G)
    Y = host(m.apex4_w4a4_gemm_mx(A6, ea, W6, ew, G))
    Aq, ea_o = omx.quantize_mx(x, G)
    Wq, ew_o = omx.quantize_mx(w, G)
    check_tolerance(Y, omx.gemm_mx_f64(Aq, ea_o, Wq, ew_o, K, G), f"mx end to end G{G}")


def test_paper_shape_sampled():
    M, N, K, G = 2048, 8192, 8192, 128
    log("mx paper shape")
    Aq, _, Wq, _ = wl.codes_workload("paper", M, N, K, G)
    r = np.random.default_rng(21)
    ea = (127 + r.integers(-4, 2, size=(M, K // G))).astype(np.uint8)
    ew = (127 + r.integers(-4, 2, size=(N, K // G))).astype(np.uint8)
    Y = gemm_from_oracle_operands(Aq, ea, Wq, ew, G)
    rows = sample_rows(M, seed=5)
    check_tolerance(Y[rows], omx.gemm_mx_f64(Aq, ea, Wq, ew, K, G, rows), "mx paper shape")


def test_group_rule_and_empty():
    import torch
    m = pk()
    x = torch.zeros((4, 256), dtype=torch.float16, device="cuda")
    with pytest.raises(m.Apex4Error):
        m.apex4_quantize_mx(x, 96)
    A6 = torch.empty((0, 96), dtype=torch.uint8, device="cuda")
    ea = torch.empty((0, 1), dtype=torch.uint8, device="cuda")
    W6 = torch.zeros((8, 96), dtype=torch.uint8, device="cuda")
    ew = torch.full((8, 1), 127, dtype=torch.uint8, device="cuda")
    assert m.apex4_w4a4_gemm_mx(A6, ea, W6, ew, 128).shape == (0, 8)
    with pytest.raises(m.Apex4Error):
        m.apex4_w4a4_gemm_mx(A6, ea, W6, ew, 256)                  # G > K


# split over K (apex4_w4a4_gemm_mx_ws): factors 4, 4, 2 and an odd M N (the
# reduction's one-element path)
MX_SPLIT = [(256, 8192, 8192, 128), (64, 1024, 2048, 32), (512, 8192, 4096, 64), (65, 1001, 2048, 128)]


@pytest.mark.parametrize("M,N,K,G", MX_SPLIT)
def test_split_k(M, N, K, G):
    import torch
    m = pk()
    need = m.apex4_w4a4_gemm_mx_workspace_size(M, N, K, G)
    log(f"mx split-K M={M} N={N} K={K} G={G} workspace={need}")
    assert need > 0 and need % (4 * M * N) == 0
    r = np.random.default_rng(M + N + K + G)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    ea = (127 + r.integers(-6, 3, size=(M, K // G))).astype(np.uint8)
    ew = (127 + r.integers(-6, 3, size=(N, K // G))).astype(np.uint8)
    d = (dev(ofp6.pack_fp6(Aq)), dev(ea), dev(ofp6.pack_fp6(Wq)), dev(ew))
    ws = torch.empty((need,), dtype=torch.uint8, device="cuda")
    Y1 = host(m.apex4_w4a4_gemm_mx_ws(*d, G, ws))
    Y2 = host(m.apex4_w4a4_gemm_mx_ws(*d, G, ws))
    assert np.array_equal(Y1.view(np.uint16), Y2.view(np.uint16))
    rows = sample_rows(M, seed=M) if M > 64 else np.arange(M)
    check_tolerance(Y1[rows], omx.gemm_mx_f64(Aq, ea, Wq, ew, K, G, rows), f"mx split {M}x{N}x{K} G{G}")
    with pytest.raises(m.Apex4Error) as e:
        m.apex4_w4a4_gemm_mx_ws(*d, G, ws[: need - 16])
    assert e.value.status == -7


def test_no_split_is_the_plain_mx_gemm():
    m = pk()
    M, N, K, G = 2048, 8192, 1024, 128
    assert m.apex4_w4a4_gemm_mx_workspace_size(M, N, K, G) == 0
    r = np.random.default_rng(9)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    ea = (127 + r.integers(-3, 3, size=(M, K // G))).astype(np.uint8)
    ew = (127 + r.integers(-3, 3, size=(N, K // G))).astype(np.uint8)
    d = (dev(ofp6.pack_fp6(Aq)), dev(ea), dev(ofp6.pack_fp6(Wq)), dev(ew))
    assert np.array_equal(host(m.apex4_w4a4_gemm_mx(*d, G)).view(np.uint16),
                          host(m.apex4_w4a4_gemm_mx_ws(*d, G)).view(np.uint16))


def test_linear_module_mx():
    """W4A4Linear(scales="mx"): weights quantized once with power-of-two scales,
    activations per call, against the oracle's MX quantize + GEMM (these row
    counts take the split-K form with the layer's own workspace)."""
    import torch
    m = pk()
    N, K, G = 1024, 2048, 64
    x, w = wl.float_workload("tiny", 64, N, K)
    lin = m.W4A4Linear(dev(w), G, scales="mx")
    Wq_o, ew_o = omx.quantize_mx(w, G)
    assert np.array_equal(host(lin.s_w), ew_o)
    assert np.array_equal(host(lin.W_q), ofp6.pack_fp6(Wq_o))
    for rows in (5, 64, 64):
        y = host(lin(dev(x[:rows]).reshape(1, rows, K)))
        assert y.shape == (1, rows, N)
        key = (rows, torch.cuda.current_stream().cuda_stream)
        assert (lin._work[key][2] is not None) == (m.apex4_w4a4_gemm_mx_workspace_size(rows, N, K, G) > 0)
        Aq_o, ea_o = omx.quantize_mx(x[:rows], G)
        check_tolerance(y[0], omx.gemm_mx_f64(Aq_o, ea_o, Wq_o, ew_o, K, G), f"mx module rows={rows}")
    with pytest.raises(ValueError):
        m.W4A4Linear(dev(w), G, scales="int8")
