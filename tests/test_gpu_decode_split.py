"""The few-row kernel's stream-K form (apex4_w4a4_gemm_ws and the other
workspace entry points, up to 32 rows).  Where round-robin tiles would leave
more than a tenth of the CUs idle and the tiles are long (below 256 tiles at
least 128 stage-groups, and K >= 24576 from 128 tiles on; K >= 24576 from 256
tiles on), the full rounds
stay round robin and the remaining tiles' (tile, stage) units are spread evenly
over the CUs; tiles are cut between workgroups, and the cut tiles' fp32 parts
are added in segment order through the workspace (Eq. group_decomposition:
splitting a group's stages changes fp32 rounding only, never the exact group
sums).

  * the plan says "decode_split" and the workspace size is positive;
  * Y within the tolerance of the oracle, and the same bits on every call and
    from a replayed graph (the counters are cleared by a kernel each call);
  * the exact group sums (debug dump with the workspace) against the oracle;
  * tiled and row-major weights give the same bits (same kernel, same cuts);
  * shapes where the round-robin form was measured faster keep it;
  * 200 back-to-back calls on one workspace, alternating two input sets, each
    give their own set's bits (the parts and counters cross XCDs through
    device-scope accesses, without a full fence);
  * seeded random few-row shapes, whichever form the plan picks, against the
    oracle in full.
"""
import numpy as np
import pytest

from parity import check_tolerance, dev, host, log
from paper_2606_08761_amd import workloads as wl

pytestmark = pytest.mark.gpu


def pk():
    import paper_2606_08761_amd as m
    return m


# (M, N, K, G): full rounds plus cut tiles at K = 24576 (a few leftover tiles
# over many workgroups, and tens of them), the mixed configuration's G = 32
# value projection (N = 1024) at M = 16 and its down projection (K = 28672) at
# M = 4, a few tiles over many stages (two tiles: fewer workgroups than CUs),
# partial last stages (K % 128 != 0, also past full rounds), per channel,
# G = 64, 256 and 512, and the 8-row form at its largest M
SHAPES = [(16, 8448, 24576, 128), (5, 9000, 24576, 128), (17, 8256, 24576, 128), (16, 1024, 8192, 32),
          (4, 1024, 28672, 32), (2, 300, 8192, 64), (32, 2048, 16384, 256), (3, 100, 16384, 128),
          (7, 1000, 4000, 32), (16, 520, 16480, 16480), (9, 64, 32768, 1024), (16, 64, 8192, 32),
          (8, 2048, 16384, 512), (3, 8448, 24608, 32)]


@pytest.mark.parametrize("M,N,K,G", SHAPES)
def test_decode_split(O, M, N, K, G):
    import torch
    m = pk()
    plan = m.apex4_w4a4_gemm_plan("gemm_ws", M, N, K, G)
    need = m.apex4_w4a4_gemm_workspace_size(M, N, K, G)
    log(f"decode split M={M} N={N} K={K} G={G}: {plan}, workspace {need} bytes")
    assert plan == ("decode_split", 1) and need > 0
    assert m.apex4_w4a4_gemm_plan("gemm", M, N, K, G) == ("decode", 1)
    r = np.random.default_rng(M * 7919 + N * 31 + K + G)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    ws = torch.empty((need,), dtype=torch.uint8, device="cuda")
    Y = m.apex4_w4a4_gemm_ws(*d, G, ws)
    Y2 = m.apex4_w4a4_gemm_ws(*d, G, ws)
    windows = [(0, M)] if M <= 8 else [(0, 3), (M - 5, 5)]
    dumps = [m.apex4_w4a4_gemm_debug(*d, G, m0, mr, workspace=ws) for m0, mr in windows]
    tiled = G >= 128 and K % 128 == 0
    Yt = m.apex4_w4a4_gemm_tiled(d[0], d[1], m.apex4_tile_weights(d[2]), d[3], G, workspace=ws) if tiled else Y
    torch.cuda.synchronize()
    assert torch.equal(Y2, Y) and torch.equal(Yt, Y)
    P_o = O.groupsums(Aq, Wq, K, G)
    for (m0, mr), (Yd, P) in zip(windows, dumps):
        assert torch.equal(Yd, Y)
        assert np.array_equal(host(P), P_o[m0:m0 + mr]), (m0, mr)
    check_tolerance(host(Y), O.gemm_rows(Aq, sa, Wq, sw, K, G), f"decode split {M}x{N}x{K} G{G}")


# round robin measured faster: the tile time is near the kernel's fixed latency
# (K = 8192 at G = 128, whatever the count of tiles; N = 10240 at G = 32; half
# the CUs busy at K = 8192, G = 32), or the last round leaves at most a tenth
# of the CUs idle (N = 8192, 57344)
KEEP = [(16, 10240, 8192, 128), (16, 1024, 8192, 128), (8, 28672, 8192, 128), (16, 10240, 8192, 32),
        (16, 8192, 28672, 32), (16, 57344, 8192, 128), (2, 300, 2048, 64), (16, 4096, 8192, 32)]


@pytest.mark.parametrize("M,N,K,G", KEEP)
def test_decode_round_robin_kept(M, N, K, G):
    m = pk()
    assert m.apex4_w4a4_gemm_plan("gemm_ws", M, N, K, G) == ("decode", 1)
    assert m.apex4_w4a4_gemm_workspace_size(M, N, K, G) == 0


def test_decode_split_graph_replay():
    """Captured calls replayed several times, with other work between the
    replays, give the eager bits each time."""
    import torch
    m = pk()
    M, N, K, G = 16, 1024, 8192, 32
    r = np.random.default_rng(5)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    ws = torch.empty((m.apex4_w4a4_gemm_workspace_size(M, N, K, G),), dtype=torch.uint8, device="cuda")
    Y = torch.empty((M, N), dtype=torch.float16, device="cuda")
    m.apex4_w4a4_gemm_ws(*d, G, ws, Y)
    torch.cuda.synchronize()
    ref = Y.clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        for _ in range(3):
            m.apex4_w4a4_gemm_ws(*d, G, ws, Y)
    torch.cuda.synchronize()
    for i in range(3):
        Y.fill_(float("nan"))
        m.apex4_w4a4_gemm(*d, G)                      # other work on the device between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y, ref), i


@pytest.mark.parametrize("M,N,K,G", [(16, 1024, 8192, 32), (5, 9000, 24576, 128), (16, 64, 8192, 32)])
def test_decode_split_many_calls(M, N, K, G):
    """Many back-to-back calls on one workspace, alternating between two input
    sets, each give the bits of their own input set.

    Each call's cut tiles are added up by whichever workgroup counts their last
    part, reading parts that other workgroups (on any XCD) wrote with
    device-scope stores.  A part read before it was written would hold the
    previous call's part, which comes from the other input set, and a stale
    counter would leave a tile unwritten or written twice; either would change
    some output of some call."""
    import torch
    m = pk()
    assert m.apex4_w4a4_gemm_plan("gemm_ws", M, N, K, G) == ("decode_split", 1)
    sets = []
    for seed in (1, 2):
        r = np.random.default_rng(M * 31 + N + K + G + seed)
        Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
        sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
        sets.append([dev(a) for a in (Aq, sa, Wq, sw)])
    ws = torch.empty((m.apex4_w4a4_gemm_workspace_size(M, N, K, G),), dtype=torch.uint8, device="cuda")
    refs = [m.apex4_w4a4_gemm(*d, G) for d in sets]   # round robin, no workspace
    refs_ws = [m.apex4_w4a4_gemm_ws(*d, G, ws) for d in sets]
    torch.cuda.synchronize()
    assert not torch.equal(refs_ws[0], refs_ws[1])
    for a, b in zip(refs, refs_ws):
        check_tolerance(host(b), host(a).astype(np.float64), f"stream-K vs round robin {M}x{N}x{K}")
    outs = [torch.empty_like(refs_ws[0]) for _ in range(200)]
    for i, Y in enumerate(outs):
        m.apex4_w4a4_gemm_ws(*sets[i & 1], G, ws, Y)
    torch.cuda.synchronize()
    bad = [i for i, Y in enumerate(outs) if not torch.equal(Y, refs_ws[i & 1])]
    assert not bad, f"{len(bad)} of {len(outs)} calls differ, first {bad[:5]}"


def _random_shapes(n=14, seed=2024):
    """Seeded (M, N, K, G) draws over the few-row range, K a multiple of G
    (not always of 128), sized so the oracle covers every output in seconds."""
    r = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        G = int(r.choice([32, 64, 128, 256, 0]))
        K = int(r.integers(32, 257)) * 64
        if G == 0:
            G = K
        K -= K % G
        if K < G:
            continue
        M, N = int(r.integers(2, 33)), int(r.integers(1, 129)) * 32 - int(r.integers(0, 32))
        if M * N * K > 1.2e9:
            continue
        out.append((M, N, K, G))
    return out


@pytest.mark.parametrize("M,N,K,G", _random_shapes())
def test_decode_workspace_random_shapes(O, M, N, K, G):
    """Random few-row shapes through the workspace entry point, whichever form
    the plan picks: every output within the tolerance of the oracle, the exact
    group sums of a row window, the same bits on a second call, and a
    workspace of at most 3 MB."""
    import torch
    m = pk()
    kern, S = m.apex4_w4a4_gemm_plan("gemm_ws", M, N, K, G)
    need = m.apex4_w4a4_gemm_workspace_size(M, N, K, G)
    log(f"random decode M={M} N={N} K={K} G={G}: {(kern, S)}, workspace {need} bytes")
    assert kern in ("decode", "decode_split") and S == 1
    assert (need > 0) == (kern == "decode_split") and need <= 3 << 20
    r = np.random.default_rng(M * 131 + N * 7 + K + G)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    ws = torch.empty((max(need, 16),), dtype=torch.uint8, device="cuda")
    Y = m.apex4_w4a4_gemm_ws(*d, G, ws)
    Y2 = m.apex4_w4a4_gemm_ws(*d, G, ws)
    m0, mr = M // 3, min(4, M - M // 3)
    Yd, P = m.apex4_w4a4_gemm_debug(*d, G, m0, mr, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(Y2, Y) and torch.equal(Yd, Y)
    assert np.array_equal(host(P), O.groupsums(Aq, Wq, K, G, m0, mr))
    check_tolerance(host(Y), O.gemm_rows(Aq, sa, Wq, sw, K, G), f"random decode {M}x{N}x{K} G{G}")
