"""apex4_w4a4_linear_ws: the quantizer, then the GEMM with the workspace entry
point's kernel choice (split over K across workgroups, or the few-row
kernel's stream-K form), the linear form of Eq. (group_decomposition) split
over K.

Checked on each shape, for row-major and (G >= 128) tiled weights:
  * the plan is the fused one-row kernel where apex4_w4a4_linear fuses, and
    apex4_w4a4_gemm_ws's (tiled: apex4_w4a4_gemm_tiled with a workspace)
    otherwise;
  * Y and the work buffers equal apex4_quantize_act followed by that GEMM
    entry point bit for bit;
  * the work buffers equal the oracle's codes and scales, and Y is within
    tolerance of the oracle on sampled rows;
  * a call that needs a workspace and gets none is refused with
    APEX4_ERR_WORKSPACE before anything is written.
"""
import ctypes

import numpy as np
import pytest

from parity import check_tolerance, dev, host, log
from paper_2606_08761_amd import workloads as wl

pytestmark = pytest.mark.gpu

# (M, N, K, G): the fused one-row linear; the stream-K few-row form (G = 32
# row-major, G = 128 on either layout); split over K at 64 and 256 rows (the
# ping-pong kernel's split at G = 128, the tile kernel's at G = 64); no split
# at 2048 rows; a K tail (K % 128 != 0)
SHAPES = [(1, 520, 8192, 128), (16, 1024, 28672, 32), (8, 1024, 28672, 128), (64, 4096, 8192, 128),
          (256, 8192, 8192, 128), (300, 2000, 4096, 64), (2048, 4096, 8192, 128), (100, 1024, 8224, 32)]

# row-major plans on a 256-CU MI355X: the stream-K few-row form, or a split over K
EXPECT = {(16, 1024, 28672, 32): "decode_split", (8, 1024, 28672, 128): "decode_split",
          (64, 4096, 8192, 128): "split", (256, 8192, 8192, 128): "split", (300, 2000, 4096, 64): "split"}


def pk():
    import paper_2606_08761_amd as m
    return m


def _rows(M):
    return np.arange(M) if M <= 64 else np.concatenate([np.arange(0, 8), np.arange(M // 2, M // 2 + 8),
                                                         np.arange(M - 8, M)])


# the tiled layout takes G >= 128
CASES = [(*s, t) for s in SHAPES for t in (False, True) if not (t and s[3] < 128)]


@pytest.mark.parametrize("M,N,K,G,tiled", CASES)
def test_linear_ws_equals_quantize_then_gemm_ws(O, M, N, K, G, tiled):
    import torch
    m = pk()
    flags = m.APEX4_DEBUG_W_TILED if tiled else 0
    plan = m.apex4_w4a4_gemm_plan("linear_ws", M, N, K, G, flags)
    ref_plan = m.apex4_w4a4_gemm_plan("linear", M, N, K, G, flags)
    log(f"linear_ws M={M} N={N} K={K} G={G} tiled={tiled}: {plan}")
    if ref_plan[0] != "fused":
        ref_plan = m.apex4_w4a4_gemm_plan("gemm_ws", M, N, K, G, flags)
    assert plan == ref_plan
    want = EXPECT.get((M, N, K, G)) if not tiled else None  # the shapes cover each workspace form
    if want == "decode_split":
        assert plan[0] == want, plan
    elif want == "split":
        assert plan[1] > 1, plan
    x = wl.activations(wl.rng_for("decode", 51, M * 3 + N + K + G), M, K)
    w = wl.weights(wl.rng_for("decode", 52, N + K + G), N, K)
    Wq, sw = m.apex4_quantize_act(dev(w), G)
    W = m.apex4_tile_weights(Wq) if tiled else Wq
    need = m.apex4_w4a4_gemm_workspace_size(M, N, K, G)
    ws = torch.empty((max(need, 16),), dtype=torch.uint8, device="cuda")
    Aw = torch.full((M, K // 2), 0xAB, dtype=torch.uint8, device="cuda")
    sw_ = torch.full((M, K // G), float("nan"), dtype=torch.float16, device="cuda")
    xd = dev(x)
    Y = m.apex4_w4a4_linear_ws(xd, W, sw, G, workspace=ws, tiled=tiled, A_q_work=Aw, s_a_work=sw_)
    Aq, sa = m.apex4_quantize_act(xd, G)
    ws2 = torch.empty_like(ws)
    if tiled:
        Y2 = m.apex4_w4a4_gemm_tiled(Aq, sa, W, sw, G, workspace=ws2)
    else:
        Y2 = m.apex4_w4a4_gemm_ws(Aq, sa, W, sw, G, workspace=ws2)
    torch.cuda.synchronize()
    assert torch.equal(Aw, Aq) and torch.equal(sw_.view(torch.int16), sa.view(torch.int16))
    assert torch.equal(Y.view(torch.int16), Y2.view(torch.int16))
    Aq_o, sa_o = O.quantize(x, G)
    Wq_o, sw_o = O.quantize(w, G)
    assert np.array_equal(host(Aq), Aq_o) and np.array_equal(host(sa).view(np.uint16), sa_o.view(np.uint16))
    rows = _rows(M)
    check_tolerance(host(Y)[rows], O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G, rows),
                    f"linear_ws {M}x{N}x{K} G{G} tiled={tiled}")


@pytest.mark.parametrize("M,N,K,G", [(16, 1024, 28672, 32), (64, 4096, 8192, 128)])
def test_linear_ws_refuses_a_missing_workspace_before_writing(M, N, K, G):
    import torch
    m = pk()
    need = m.apex4_w4a4_gemm_workspace_size(M, N, K, G)
    assert need > 0
    x = torch.ones((M, K), dtype=torch.float16, device="cuda")
    Wq = torch.zeros((N, K // 2), dtype=torch.uint8, device="cuda")
    sw = torch.ones((N, K // G), dtype=torch.float16, device="cuda")
    Y = torch.full((M, N), 7.0, dtype=torch.float16, device="cuda")
    Aw = torch.full((M, K // 2), 0xAB, dtype=torch.uint8, device="cuda")
    sa = torch.full((M, K // G), 3.0, dtype=torch.float16, device="cuda")
    ws = torch.empty((need,), dtype=torch.uint8, device="cuda")
    L = m.lib()
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for wsp, nbytes in ((ctypes.c_void_p(0), 0), (P(ws), need - 16)):
        rc = L.apex4_w4a4_linear_ws(P(x), P(Wq), P(sw), M, N, K, G, P(Y), P(Aw), P(sa), wsp, nbytes, 0, stream)
        assert rc == -7, rc
    torch.cuda.synchronize()
    assert bool((Aw == 0xAB).all()) and bool((sa == 3.0).all()) and bool((Y == 7.0).all())


@pytest.mark.parametrize("tiled", [False, True])
def test_linear_ws_zero_and_two_rows(O, tiled):
    """M = 0 is a no-op; M = 2 (the dot-product kernel on tiled weights, the
    few-row kernel on row-major ones) equals the quantizer plus that GEMM."""
    import torch
    m = pk()
    N, K, G = 264, 4096, 128
    w = wl.weights(wl.rng_for("decode", 53, N + K), N, K)
    Wq, sw = m.apex4_quantize_act(dev(w), G)
    W = m.apex4_tile_weights(Wq) if tiled else Wq
    Y0 = m.apex4_w4a4_linear_ws(torch.empty((0, K), dtype=torch.float16, device="cuda"), W, sw, G, tiled=tiled)
    assert Y0.shape == (0, N)
    x = wl.activations(wl.rng_for("decode", 54, K), 2, K)
    xd = dev(x)
    Y = m.apex4_w4a4_linear_ws(xd, W, sw, G, tiled=tiled)
    Aq, sa = m.apex4_quantize_act(xd, G)
    Y2 = m.apex4_w4a4_gemm_tiled(Aq, sa, W, sw, G) if tiled else m.apex4_w4a4_gemm_ws(Aq, sa, W, sw, G)
    torch.cuda.synchronize()
    assert torch.equal(Y.view(torch.int16), Y2.view(torch.int16))
    Aq_o, sa_o = O.quantize(x, G)
    Wq_o, sw_o = O.quantize(w, G)
    check_tolerance(host(Y), O.gemm_rows(Aq_o, sa_o, Wq_o, sw_o, K, G), f"linear_ws 2 rows tiled={tiled}")
