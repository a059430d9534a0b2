"""Exact integer group sums from the kernels that compute Y (APEX4 Sec. 3.2.1,
Eq. group_decomposition: P[m, n, g] = sum_{k in g} A_q[m, k] W_q[n, k]).

Every check here goes through the debug entry points, which run the same
kernel choice as the production call and return, from the same launches, Y
and the exact int32 group sums of a row window:

  * P is bit-identical to the oracle's int64 sums, computed from the oracle's
    own quantization of the same binary16 inputs (the device codes are checked
    equal to the oracle's first);
  * the debug Y is bit-identical to the production entry point's Y;
  * apex4_w4a4_gemm_plan names the kernel that ran, and the test asserts the
    one that the workload is meant to exercise (the ping-pong kernel at the
    paper shape, the streaming and one-row kernels at decode sizes, the split
    path where the workspace entry point splits).

Workloads: the tiny case and the paper shape (M=2048, N=K=8192, G=128; all
rows of Y, and P over all rows in windows of 256), the Llama-2-70B linears at
M in {16, 256, 4096}, the granularity sweep (M=4096, N=K=8192) and the decode
linears (M in {1, 8, 32}).  The G = 128 ping-pong kernel is also checked bit
for bit against the general tile kernel.
"""
import numpy as np
import pytest

from parity import check_tolerance, dev, host, log
from paper_2606_08761_amd import workloads as wl

pytestmark = pytest.mark.gpu


def pk():
    import paper_2606_08761_amd as m
    return m


def windows(M):
    """Row windows: row 0, both sides of the 128-row tile boundaries, the middle, the end."""
    if M <= 32:
        return [(0, M)]
    out = [(0, 4), (126, 4), (M // 2 - 2, 4), (M - 4, 4)]
    return sorted(set((m0, mr) for m0, mr in out if 0 <= m0 and m0 + mr <= M))


def workspace(M, N, K, G):
    import torch
    need = pk().apex4_w4a4_gemm_workspace_size(M, N, K, G)
    return torch.empty((max(need, 16),), dtype=torch.uint8, device="cuda"), need


# ---------------------------------------------------------------- paper shape


@pytest.fixture(scope="module")
def paper():
    """The paper-shape codes workload, on both sides, and the production Y."""
    import torch
    M, N, K, G = 2048, 8192, 8192, 128
    log("paper shape: generate")
    Aq, sa, Wq, sw = wl.codes_workload("paper", M, N, K, G)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    Y = pk().apex4_w4a4_gemm(*d, G)
    torch.cuda.synchronize()
    yield dict(M=M, N=N, K=K, G=G, host=(Aq, sa, Wq, sw), dev=d, Y=Y)
    del d, Y
    torch.cuda.empty_cache()


def test_paper_shape_plan(paper):
    m = pk()
    assert m.apex4_w4a4_gemm_plan("gemm", 2048, 8192, 8192, 128) == ("pingpong", 1)
    assert m.apex4_w4a4_gemm_plan("gemm", 2048, 8192, 8192, 128, m.APEX4_DEBUG_GENERAL_TILES) == ("tile128", 1)


def test_paper_shape_full_y(O, paper):
    """Every one of the 2048 x 8192 outputs against the oracle's binary64 y."""
    Aq, sa, Wq, sw = paper["host"]
    Y = host(paper["Y"])
    for r0 in range(0, paper["M"], 512):
        rows = np.arange(r0, r0 + 512)
        log(f"paper shape: full Y rows {r0}..{r0 + 511}")
        check_tolerance(Y[rows], O.gemm_rows(Aq, sa, Wq, sw, paper["K"], paper["G"], rows), f"paper rows {r0}+")


@pytest.mark.parametrize("m0", list(range(0, 2048, 256)))
def test_paper_shape_groupsums_pingpong(O, paper, m0):
    """P of rows [m0, m0 + 256) from the ping-pong kernel (all rows over the eight cases)."""
    import torch
    m = pk()
    Aq, sa, Wq, sw = paper["host"]
    K, G, mr = paper["K"], paper["G"], 256
    log(f"paper shape: P rows {m0}..{m0 + mr - 1}")
    Yd, P = m.apex4_w4a4_gemm_debug(*paper["dev"], G, m0, mr)
    torch.cuda.synchronize()
    assert torch.equal(Yd, paper["Y"])
    Pd = host(P)
    del P
    assert np.array_equal(Pd, O.groupsums(Aq, Wq, K, G, m0, mr))


def test_pingpong_equals_general_tiles(O, paper):
    """The ping-pong schedule changes when work is issued, not the arithmetic:
    the same Y and P bits as the general 128 x 256 tile kernel (also at G = 256,
    where its group spans two stages, on the shapes below)."""
    import torch
    m = pk()
    G = paper["G"]
    Yg, Pg = m.apex4_w4a4_gemm_debug(*paper["dev"], G, 1020, 8, flags=m.APEX4_DEBUG_GENERAL_TILES)
    Yp, Pp = m.apex4_w4a4_gemm_debug(*paper["dev"], G, 1020, 8)
    torch.cuda.synchronize()
    assert torch.equal(Yg, paper["Y"]) and torch.equal(Yp, paper["Y"])
    assert torch.equal(Pg, Pp)


# ragged shapes on 128 x 256 tiles (G = 128, and G = 256: two stages per
# group), and split-K shapes (G = 128)
PP_SHAPES = [(1111, 8200, 640, 128), (1500, 8195, 1152, 128), (2050, 4100, 4096, 128), (4096, 4096, 1024, 128),
             (1111, 8200, 1280, 256), (2050, 4100, 4096, 256), (4096, 4096, 512, 256), (2048, 4096, 28672, 256)]
PP_SPLIT = [(256, 8192, 8192, 128), (512, 4096, 8192, 128), (300, 2000, 4096, 128)]


@pytest.mark.parametrize("M,N,K,G", PP_SHAPES + PP_SPLIT)
def test_pingpong_equals_general_tiles_shapes(O, M, N, K, G):
    import torch
    m = pk()
    split = (M, N, K, G) in PP_SPLIT
    entry = "gemm_ws" if split else "gemm"
    kern, S = m.apex4_w4a4_gemm_plan(entry, M, N, K, G)
    log(f"pp vs general {M}x{N}x{K}: {kern} S={S}")
    assert kern == "pingpong"
    assert (S > 1) == split
    r = np.random.default_rng(M * 31 + N * 7 + K)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    ws = workspace(M, N, K, G)[0] if split else None
    m0 = min(126, M - 4)
    Yp, Pp = m.apex4_w4a4_gemm_debug(*d, G, m0, 4, workspace=ws)
    Yg, Pg = m.apex4_w4a4_gemm_debug(*d, G, m0, 4, workspace=ws, flags=m.APEX4_DEBUG_GENERAL_TILES)
    Y = m.apex4_w4a4_gemm_ws(*d, G, ws) if split else m.apex4_w4a4_gemm(*d, G)
    torch.cuda.synchronize()
    assert torch.equal(Yp, Y) and torch.equal(Yg, Y)
    assert torch.equal(Pp, Pg)
    assert np.array_equal(host(Pp), O.groupsums(Aq, Wq, K, G, m0, 4))


def test_tiny_groupsums_every_path(O):
    """The tiny workload in full through gemm, gemm_ws and the general tiles."""
    import torch
    m = pk()
    M, N, K, G = 64, 1024, 1024, 128
    Aq, sa, Wq, sw = wl.codes_workload("tiny", M, N, K, G)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    P_o = O.groupsums(Aq, Wq, K, G)
    ws = workspace(M, N, K, G)[0]
    Y = m.apex4_w4a4_gemm(*d, G)
    Yws = m.apex4_w4a4_gemm_ws(*d, G, ws)
    for kw, Yref in ((dict(), Y), (dict(workspace=ws), Yws), (dict(flags=m.APEX4_DEBUG_GENERAL_TILES), None)):
        Yd, P = m.apex4_w4a4_gemm_debug(*d, G, **kw)
        torch.cuda.synchronize()
        if Yref is not None:
            assert torch.equal(Yd, Yref), kw
        assert np.array_equal(host(P), P_o), kw
    assert np.array_equal(host(m.apex4_w4a4_gemm_groupsums(d[0], d[2], G)), P_o)


# ------------------------------------------------------- float workloads


class Quantized:
    """A binary16 matrix quantized on the device and by the oracle, codes and
    scales checked equal in full."""

    def __init__(self, O, x, G):
        m = pk()
        self.x = x
        self.q_d, self.s_d = m.apex4_quantize_act(dev(x), G)
        self.q_o, self.s_o = O.quantize(x, G)
        assert np.array_equal(host(self.q_d), self.q_o)
        assert np.array_equal(host(self.s_d).view(np.uint16), self.s_o.view(np.uint16))


def _linear_case(O, name, W, x, G, M):
    """P windows through apex4_w4a4_linear_debug and apex4_w4a4_gemm_debug (with
    the workspace entry point's kernel choice), both against the oracle, for
    row-major and tiled weights (M >= 2: the same Y bits from either)."""
    import torch
    m = pk()
    N, K = W.q_o.shape[0], x.shape[1]
    A = Quantized(O, x, G)
    ws, need = workspace(M, N, K, G)
    plan_lin = m.apex4_w4a4_gemm_plan("linear", M, N, K, G)
    plan_ws = m.apex4_w4a4_gemm_plan("gemm_ws", M, N, K, G)
    log(f"{name}: linear {plan_lin}, gemm_ws {plan_ws}")
    xd = dev(x)
    Wt = m.apex4_tile_weights(W.q_d)
    T = m.APEX4_DEBUG_W_TILED
    Y_lin = m.apex4_w4a4_linear(xd, W.q_d, W.s_d, G)
    Y_ws = m.apex4_w4a4_gemm_ws(A.q_d, A.s_d, W.q_d, W.s_d, G, ws)
    Y_lin_t = m.apex4_w4a4_linear_tiled(xd, Wt, W.s_d, G)
    Y_ws_t = m.apex4_w4a4_gemm_tiled(A.q_d, A.s_d, Wt, W.s_d, G, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(Y_lin_t, Y_lin) and torch.equal(Y_ws_t, Y_ws), name
    for m0, mr in windows(M):
        P_o = O.groupsums(A.q_o, W.q_o, K, G, m0, mr)
        Yl, Aw, sw_, Pl = m.apex4_w4a4_linear_debug(xd, W.q_d, W.s_d, G, m0, mr)
        Yw, Pw = m.apex4_w4a4_gemm_debug(A.q_d, A.s_d, W.q_d, W.s_d, G, m0, mr, workspace=ws)
        Ylt, _, _, Plt = m.apex4_w4a4_linear_debug(xd, Wt, W.s_d, G, m0, mr, flags=T)
        Ywt, Pwt = m.apex4_w4a4_gemm_debug(A.q_d, A.s_d, Wt, W.s_d, G, m0, mr, workspace=ws, flags=T)
        torch.cuda.synchronize()
        assert torch.equal(Yl, Y_lin) and torch.equal(Ylt, Y_lin), (name, m0)
        assert torch.equal(Yw, Y_ws) and torch.equal(Ywt, Y_ws), (name, m0)
        assert torch.equal(Aw, A.q_d) and torch.equal(sw_.view(torch.int16), A.s_d.view(torch.int16))
        for tag, Pd in (("linear", Pl), ("gemm_ws", Pw), ("linear tiled", Plt), ("gemm_ws tiled", Pwt)):
            assert np.array_equal(host(Pd), P_o), (name, tag, m0, mr)
    rows = np.unique(np.concatenate([np.arange(w0, w0 + wr) for w0, wr in windows(M)]))
    y = O.gemm_rows(A.q_o, A.s_o, W.q_o, W.s_o, K, G, rows)
    check_tolerance(host(Y_lin)[rows], y, f"{name} linear")
    check_tolerance(host(Y_ws)[rows], y, f"{name} gemm_ws")
    return plan_lin, plan_ws


@pytest.mark.parametrize("linear", list(wl.LLAMA70B_LINEARS))
def test_llama70b_linear_groupsums(O, linear):
    N, K = wl.LLAMA70B_LINEARS[linear]
    G = 128
    log(f"llama70b {linear}: weights {N}x{K}")
    W = Quantized(O, wl.weights(wl.rng_for("llama70b", 10 + list(wl.LLAMA70B_LINEARS).index(linear)), N, K), G)
    kernels = set()
    for M in (16, 256, 4096):
        x = wl.activations(wl.rng_for("llama70b", 20, M * 100 + K // 1024), M, K)
        lin, ws = _linear_case(O, f"{linear} M={M}", W, x, G, M)
        kernels.update((lin[0], ws[0]))
        if M == 16:  # the workspace entry takes the stream-K form where round robin leaves CUs idle
            assert lin == ("decode", 1) and ws in (("decode", 1), ("decode_split", 1))
        if M == 4096:
            assert lin == ("pingpong", 1)
    log(f"llama70b {linear}: kernels {sorted(kernels)}")


@pytest.mark.parametrize("G", [128, 256, 512, 8192])
def test_granularity_sweep_groupsums(O, G):
    import torch
    m = pk()
    M, N, K = 4096, 8192, 8192
    log(f"gsweep G={G}")
    W = Quantized(O, wl.weights(wl.rng_for("gsweep", 2), N, K), G)
    x = wl.activations(wl.rng_for("gsweep", 1, G), M, K)
    A = Quantized(O, x, G)
    kern = m.apex4_w4a4_gemm_plan("gemm", M, N, K, G)
    assert kern == (("pingpong" if G in (128, 256) else "tile128"), 1)
    Y = m.apex4_w4a4_gemm(A.q_d, A.s_d, W.q_d, W.s_d, G)
    for m0, mr in windows(M):
        Yd, P = m.apex4_w4a4_gemm_debug(A.q_d, A.s_d, W.q_d, W.s_d, G, m0, mr)
        torch.cuda.synchronize()
        assert torch.equal(Yd, Y)
        assert np.array_equal(host(P), O.groupsums(A.q_o, W.q_o, K, G, m0, mr)), (G, m0)


@pytest.mark.parametrize("N,K", [(8192, 8192), (28672, 8192)])
def test_decode_linear_groupsums(O, N, K):
    """Decode sizes: every row's P, through the linear (fused one-row kernel
    where it applies) and the GEMM entry points."""
    import torch
    m = pk()
    G = 128
    W = Quantized(O, wl.weights(wl.rng_for("decode", 2, N), N, K), G)
    for M in (1, 8, 32):
        x = wl.activations(wl.rng_for("decode", 1, M * 1000 + N // 1024), M, K)
        A = Quantized(O, x, G)
        plan = m.apex4_w4a4_gemm_plan("linear", M, N, K, G)
        log(f"decode N={N} K={K} M={M}: {plan}")
        assert plan[0] == ("decode" if M > 1 else ("fused" if N * K <= 8192 * 8192 else "gemv"))
        P_o = O.groupsums(A.q_o, W.q_o, K, G)
        Y = m.apex4_w4a4_linear(dev(x), W.q_d, W.s_d, G)
        Yl, _, _, Pl = m.apex4_w4a4_linear_debug(dev(x), W.q_d, W.s_d, G)
        Yg, Pg = m.apex4_w4a4_gemm_debug(A.q_d, A.s_d, W.q_d, W.s_d, G)
        # the tiled layout: the same kernels' tiled forms
        Wt = m.apex4_tile_weights(W.q_d)
        T = m.APEX4_DEBUG_W_TILED
        log(f"decode N={N} K={K} M={M} tiled: {m.apex4_w4a4_gemm_plan('linear', M, N, K, G, T)}")
        Yt = m.apex4_w4a4_linear_tiled(dev(x), Wt, W.s_d, G)
        Ylt, _, _, Plt = m.apex4_w4a4_linear_debug(dev(x), Wt, W.s_d, G, flags=T)
        Ygt, Pgt = m.apex4_w4a4_gemm_debug(A.q_d, A.s_d, Wt, W.s_d, G, flags=T)
        torch.cuda.synchronize()
        assert torch.equal(Yl, Y) and torch.equal(Yg, Y)
        assert torch.equal(Ylt, Yt) and torch.equal(Ygt, Yt)
        if M > 1:
            assert torch.equal(Yt, Y)
        for Pd in (Pl, Pg, Plt, Pgt):
            assert np.array_equal(host(Pd), P_o)
        y = O.gemm_rows(A.q_o, A.s_o, W.q_o, W.s_o, K, G)
        check_tolerance(host(Y), y, f"decode M={M}")
        check_tolerance(host(Yt), y, f"decode tiled M={M}")


# the decode and one-row kernels at every G, sub-group partials (G > 128) included
DECODE_G = [(1, 1000, 8192, 32), (1, 257, 2048, 1024), (1, 300, 3072, 3072), (5, 40, 2560, 512),
            (32, 300, 1536, 1536), (16, 64, 28672, 256), (4, 300, 2048, 64), (32, 1024, 1024, 32),
            (8, 520, 8192, 1024), (1, 520, 4096, 64)]


@pytest.mark.parametrize("M,N,K,G", DECODE_G)
def test_decode_kernels_groupsums(O, M, N, K, G):
    import torch
    m = pk()
    plan = m.apex4_w4a4_gemm_plan("gemm", M, N, K, G)
    log(f"decode kernels {M}x{N}x{K} G={G}: {plan}")
    assert plan[0] == ("gemv" if M == 1 else "decode")
    r = np.random.default_rng(M * 104729 + N * 13 + K + G)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    Y = m.apex4_w4a4_gemm(*d, G)
    Yd, P = m.apex4_w4a4_gemm_debug(*d, G)
    P2 = m.apex4_w4a4_gemm_groupsums(d[0], d[2], G)
    torch.cuda.synchronize()
    assert torch.equal(Yd, Y)
    P_o = O.groupsums(Aq, Wq, K, G)
    assert np.array_equal(host(P), P_o)
    assert np.array_equal(host(P2), P_o)


# Shapes where the few-row kernel stages the activations in LDS (K % 512 == 0,
# the M packed rows beside the scales within 144 KB, and each wave walking at
# least 16 stages: ceil(tiles / CUs) * ceil(K / 1024) >= 16 on 256 CUs), at
# every group kind: 32 and 64 (several groups per stage), 128, 256 (sums over
# two stages), per channel, and an odd row count.
DECODE_ALDS = [(4, 300, 32768, 64), (8, 9000, 8192, 32), (16, 600, 16384, 256), (32, 8300, 8192, 8192),
               (3, 20000, 8192, 128), (32, 28672, 8192, 128)]


@pytest.mark.parametrize("M,N,K,G", DECODE_ALDS)
def test_decode_staged_activations(O, M, N, K, G):
    import torch
    m = pk()
    tiles, stages = -(-N // 32), -(-K // 1024)
    a_lds = -(-M * K // 2 // 1024) * 1024
    assert K % 512 == 0 and a_lds + 2 * (K // G) * 64 <= 144 * 1024 and -(-tiles // 256) * stages >= 16
    plan = m.apex4_w4a4_gemm_plan("gemm", M, N, K, G)
    log(f"decode staged activations {M}x{N}x{K} G={G}: {plan}")
    assert plan[0] == "decode"
    r = np.random.default_rng(M * 7919 + N * 17 + K + G)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    Y = m.apex4_w4a4_gemm(*d, G)
    Yd, P = m.apex4_w4a4_gemm_debug(*d, G)
    P2 = m.apex4_w4a4_gemm_groupsums(d[0], d[2], G)
    Yt = m.apex4_w4a4_gemm_tiled(d[0], d[1], m.apex4_tile_weights(d[2]), d[3], G) if G >= 128 else Y
    torch.cuda.synchronize()
    assert torch.equal(Yd, Y) and torch.equal(Yt, Y)
    P_o = O.groupsums(Aq, Wq, K, G)
    assert np.array_equal(host(P), P_o)
    assert np.array_equal(host(P2), P_o)
    check_tolerance(host(Y), O.gemm_rows(Aq, sa, Wq, sw, K, G), f"decode staged {M}x{N}x{K} G{G}")
