"""apex4_w4a4_gemm_noalloc: the workspace GEMM with the library's static
per-device scratch in place of a caller workspace (for callers that cannot
allocate).  Its Y must equal apex4_w4a4_gemm_ws's bit for bit (same kernels,
same split or stream-K cuts), and the oracle's within tolerance, on
consecutive calls that share the scratch, the second with a smaller problem (a
stale partial or counter from the first call would show up in it), and
captured in a graph whose replays, with eager calls between, give the eager
bits.
"""
import numpy as np
import pytest

from parity import check_tolerance, dev, host, log
from paper_2606_08761_amd import workloads as wl

pytestmark = pytest.mark.gpu

# (M, N, K, G): each pair is a larger split then a smaller one.  The first
# needs the whole scratch on a 256-CU device (4 x 256 x 8192 fp32 partials).
PAIRS = [
    ((256, 8192, 8192, 128), (300, 2000, 4096, 128)),
    ((128, 2048, 8192, 32), (65, 1001, 2048, 32)),
    ((256, 4096, 8192, 8192), (64, 520, 3072, 3072)),
    ((300, 2000, 4096, 128), (16, 1024, 4096, 128)),   # then a shape that does not split
    ((16, 1024, 8192, 32), (4, 64, 28672, 32)),        # the few-row kernel's stream-K form twice
]


def _case(O, M, N, K, G, seed):
    import torch
    m = pk()
    r = np.random.default_rng(seed)
    Aq, Wq = wl.random_codes(r, M, K), wl.random_codes(r, N, K)
    sa, sw = wl.random_scales(r, M, K // G), wl.random_scales(r, N, K // G)
    d = [dev(a) for a in (Aq, sa, Wq, sw)]
    need = m.apex4_w4a4_gemm_workspace_size(M, N, K, G)
    assert need <= m.APEX4_NOALLOC_SCRATCH_BYTES
    plan = m.apex4_w4a4_gemm_plan("gemm_ws", M, N, K, G)
    log(f"noalloc M={M} N={N} K={K} G={G}: {plan}, workspace {need} bytes")
    Y = m.apex4_w4a4_gemm_noalloc(*d, G)
    ws = torch.empty((max(need, 16),), dtype=torch.uint8, device="cuda")
    Y_ws = m.apex4_w4a4_gemm_ws(*d, G, ws)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y_ws), (M, N, K, G)
    rows = np.unique(np.concatenate([np.arange(min(M, 4)), np.arange(M - 2, M), r.integers(0, M, size=6)]))
    check_tolerance(host(Y)[rows], O.gemm_rows(Aq, sa, Wq, sw, K, G, rows), f"noalloc {M}x{N}x{K} G{G}")
    return plan


def pk():
    import paper_2606_08761_amd as m
    return m


@pytest.mark.parametrize("first,second", PAIRS)
def test_noalloc_matches_workspace_entry(O, first, second):
    p1 = _case(O, *first, seed=sum(first))
    p2 = _case(O, *second, seed=sum(second) + 1)
    uses_ws = lambda p: p[1] > 1 or p[0] == "decode_split"  # noqa: E731
    assert uses_ws(p1)
    if second != (16, 1024, 4096, 128):
        assert uses_ws(p2)


def test_noalloc_repeat_and_empty():
    """Back-to-back calls on one stream give the same bits; M == 0 is a no-op."""
    import torch
    m = pk()
    M, N, K, G = 256, 8192, 8192, 128
    r = np.random.default_rng(7)
    d = [dev(a) for a in (wl.random_codes(r, M, K), wl.random_scales(r, M, K // G),
                          wl.random_codes(r, N, K), wl.random_scales(r, N, K // G))]
    Y1 = m.apex4_w4a4_gemm_noalloc(*d, G)
    Y2 = m.apex4_w4a4_gemm_noalloc(*d, G)
    torch.cuda.synchronize()
    assert torch.equal(Y1, Y2)
    m.apex4_w4a4_gemm_noalloc(d[0][:0], d[1][:0], d[2], d[3], G)
    torch.cuda.synchronize()


def test_noalloc_graph_replay():
    """The entry point's use case: captured in a graph (split over K, and the
    few-row kernel's stream-K form, both on the static scratch), replayed
    three times with eager calls between; every replay gives the eager bits."""
    import torch
    m = pk()
    cases = [(256, 8192, 8192, 128), (16, 1024, 8192, 32)]
    ins, eager = [], []
    for (M, N, K, G) in cases:
        r = np.random.default_rng(M + N + K + G)
        d = [dev(a) for a in (wl.random_codes(r, M, K), wl.random_scales(r, M, K // G),
                              wl.random_codes(r, N, K), wl.random_scales(r, N, K // G))]
        ins.append(d)
        eager.append(m.apex4_w4a4_gemm_noalloc(*d, G))
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        outs = [m.apex4_w4a4_gemm_noalloc(*d, c[3]) for d, c in zip(ins, cases)]
    torch.cuda.synchronize()
    for i in range(3):
        for y in outs:
            y.fill_(float("nan"))
        for d, c in zip(ins, cases):                 # eager calls on the same scratch between replays
            m.apex4_w4a4_gemm_noalloc(*d, c[3])
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for y, e in zip(outs, eager):
            assert torch.equal(y, e), i
