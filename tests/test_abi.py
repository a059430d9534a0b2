"""Host-side checks of the C ABI (no GPU needed, no kernel launched).

  * libapex4.so loads and exports every function include/apex4.h declares;
  * argument validation returns the documented status codes before any HIP
    call (pointers passed here are host addresses that must never be touched);
  * the Python binding refuses non-device tensors instead of falling back.
"""
import ctypes
import os
import re
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "apex4.h")


@pytest.fixture(scope="module")
def L():
    import paper_2606_08761_amd as pk
    if not os.path.exists(pk.LIB_PATH):
        from paper_2606_08761_amd import build
        build.build()
    return pk.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(apex4_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for f in ("apex4_quantize_act", "apex4_w4a4_gemm", "apex4_w4a4_gemm_groupsums", "apex4_w4a4_gemm_debug",
              "apex4_w4a4_gemm_plan", "apex4_w4a4_linear", "apex4_w4a4_linear_debug", "apex4_pack_fp6", "apex4_w4a4_gemm_fp6", "apex4_w4a4_gemm_workspace_size",
              "apex4_w4a4_gemm_ws", "apex4_quantize_mx", "apex4_w4a4_gemm_mx", "apex4_w4a4_gemm_mx_workspace_size",
              "apex4_w4a4_gemm_mx_ws", "apex4_status_string", "apex4_version"):
        assert f in names


def test_library_exports_every_declared_symbol(L):
    import paper_2606_08761_amd as pk
    out = subprocess.run(["nm", "-D", "--defined-only", pk.LIB_PATH], capture_output=True, text=True, check=True)
    exported = set(re.findall(r"\bT (apex4_\w+)", out.stdout))
    for f in declared_functions():
        assert f in exported, f
        assert hasattr(L, f)
    assert set(pk.EXPORTED) <= exported


def test_status_strings(L):
    for code, name in {0: "APEX4_OK", -1: "APEX4_ERR_NULL", -2: "APEX4_ERR_SHAPE", -3: "APEX4_ERR_GROUP",
                       -4: "APEX4_ERR_ALIGN", -5: "APEX4_ERR_LAUNCH", -6: "APEX4_ERR_DEVICE"}.items():
        assert L.apex4_status_string(code).decode().startswith(name)
    assert L.apex4_status_string(-7).decode().startswith("APEX4_ERR_WORKSPACE")
    assert L.apex4_status_string(12345)
    assert L.apex4_version() >= 200


class Host:
    """16-byte aligned host buffers whose addresses stand in for device pointers.
    Validation fails before anything dereferences them."""

    def __init__(self):
        self.buf = np.zeros(4096, np.uint8)
        base = self.buf.ctypes.data
        self.p = (base + 15) & ~15

    def ptr(self, off=0):
        return ctypes.c_void_p(self.p + off)


NULL = ctypes.c_void_p(0)


def test_quantize_validation(L):
    h = Host()
    q = L.apex4_quantize_act
    s = NULL
    assert q(NULL, 4, 256, 128, h.ptr(), h.ptr(), s) == -1
    assert q(h.ptr(), 4, 256, 128, NULL, h.ptr(), s) == -1
    assert q(h.ptr(), 4, 256, 128, h.ptr(), NULL, s) == -1
    assert q(h.ptr(), -1, 256, 128, h.ptr(), h.ptr(), s) == -2
    assert q(h.ptr(), 4, 80, 16, h.ptr(), h.ptr(), s) == -2        # K % 32
    assert q(h.ptr(), 4, 16, 16, h.ptr(), h.ptr(), s) == -2        # K < 32
    assert q(h.ptr(), 4, 0, 128, h.ptr(), h.ptr(), s) == -2
    # K % 32 == 0 and any G % 32 == 0 dividing K pass the shape and group
    # rules: the misaligned x is the first error
    for K, G in ((32, 32), (96, 32), (96, 96), (160, 160), (8224, 32), (480, 160), (65568, 65568)):
        assert q(h.ptr(8), 4, K, G, h.ptr(), h.ptr(), s) == -4, (K, G)
    assert q(h.ptr(), 4, 256, 48, h.ptr(), h.ptr(), s) == -3       # G % 32
    assert q(h.ptr(), 4, 256, 512, h.ptr(), h.ptr(), s) == -3      # G > K
    assert q(h.ptr(), 4, 384, 256, h.ptr(), h.ptr(), s) == -2      # K % G
    assert q(h.ptr(), 4, 256, 0, h.ptr(), h.ptr(), s) == -3
    assert q(h.ptr(8), 4, 256, 128, h.ptr(), h.ptr(), s) == -4
    assert q(h.ptr(), 4, 256, 128, h.ptr(2), h.ptr(), s) == -4
    assert q(h.ptr(), 4, 256, 128, h.ptr(), h.ptr(4), s) == -4


def test_gemm_validation(L):
    h = Host()
    g = L.apex4_w4a4_gemm
    s = NULL
    ok = [h.ptr()] * 4
    assert g(NULL, *ok[1:], 4, 8, 256, 128, h.ptr(), s) == -1
    assert g(*ok, 4, 8, 256, 128, NULL, s) == -1
    assert g(*ok, -1, 8, 256, 128, h.ptr(), s) == -2
    assert g(*ok, 4, 0, 256, 128, h.ptr(), s) == -2
    assert g(*ok, 4, 8, 16, 16, h.ptr(), s) == -2                  # K < 32
    assert g(*ok, 4, 8, 48, 48, h.ptr(), s) == -2                  # K % 32
    assert g(*ok, 4, 8, 200, 200, h.ptr(), s) == -2
    # K >= 32, K % 32 == 0 with G in {32, ..., 1024} dividing K or G == K <= 65536
    # pass the shape and group rules (the misaligned A_q is the first error)
    for K, G in ((32, 32), (64, 64), (96, 32), (96, 96), (160, 32), (160, 160), (320, 64), (8224, 32),
                 (8224, 8224), (65536, 65536), (16352, 32)):
        assert g(h.ptr(1), *ok[1:], 4, 8, K, G, h.ptr(), s) == -4, (K, G)
    assert g(*ok, 4, 8, 65568, 65568, h.ptr(), s) == -3            # per-channel K above 65536
    assert g(*ok, 4, 8, 131072, 131072, h.ptr(), s) == -3
    assert g(*ok, 4, 8, 96, 64, h.ptr(), s) == -2                  # K % G
    assert g(*ok, 4, 8, 384, 96, h.ptr(), s) == -3                 # G not in {32,...,1024} and not K
    assert g(*ok, 4, 8, 4096, 2048, h.ptr(), s) == -3
    assert g(*ok, 4, 8, 1024, 1000, h.ptr(), s) == -3
    assert g(*ok, 4, 8, 384, 256, h.ptr(), s) == -2                # K % G
    assert g(*ok, 1 << 20, 8, 1 << 13, 128, h.ptr(), s) == -2      # A_q of 4 GiB
    assert g(*ok, 4, 1 << 21, 1 << 12, 128, h.ptr(), s) == -2      # W_q of 4 GiB
    assert g(h.ptr(1), *ok[1:], 4, 8, 256, 128, h.ptr(), s) == -4
    assert g(*ok, 4, 8, 256, 128, h.ptr(2), s) == -4


def test_groupsums_validation(L):
    h = Host()
    f = L.apex4_w4a4_gemm_groupsums
    s = NULL
    assert f(NULL, h.ptr(), 8, 8, 256, 128, 0, 8, h.ptr(), s) == -1
    assert f(h.ptr(), h.ptr(), 8, 8, 256, 128, 0, 8, NULL, s) == -1
    assert f(h.ptr(), h.ptr(), 8, 8, 256, 128, 4, 5, h.ptr(), s) == -2   # window past M
    assert f(h.ptr(), h.ptr(), 8, 8, 256, 128, -1, 2, h.ptr(), s) == -2
    assert f(h.ptr(), h.ptr(), 8, 8, 256, 96, 0, 8, h.ptr(), s) == -3
    assert f(h.ptr(), h.ptr(), 8, 8, 256, 128, 0, 8, h.ptr(4), s) == -4


def test_debug_validation(L):
    h = Host()
    f = L.apex4_w4a4_gemm_debug
    s = NULL
    ok = [h.ptr()] * 4
    ws = (NULL, 0)
    assert f(*ok, 8, 8, 256, 128, h.ptr(), *ws, 0, 8, NULL, 0, s) == -1       # no P for a window
    assert f(*ok, 8, 8, 256, 128, NULL, *ws, 0, 8, h.ptr(), 0, s) == -1       # no Y
    assert f(*ok, 8, 8, 256, 128, h.ptr(), *ws, 4, 5, h.ptr(), 0, s) == -2    # window past M
    assert f(*ok, 8, 8, 256, 128, h.ptr(), *ws, 0, 8, h.ptr(), 4, s) == -2    # unknown flag
    assert f(*ok, 8, 8, 256, 96, h.ptr(), *ws, 0, 8, h.ptr(), 0, s) == -3
    assert f(*ok, 8, 8, 256, 128, h.ptr(), *ws, 0, 8, h.ptr(4), 0, s) == -4   # misaligned P
    assert f(*ok, 8, 8, 256, 128, h.ptr(), h.ptr(8), 1 << 20, 0, 8, h.ptr(), 0, s) == -4
    g = L.apex4_w4a4_linear_debug
    args = [h.ptr()] * 3
    assert g(*args, 4, 8, 256, 128, h.ptr(), h.ptr(), h.ptr(), 0, 4, NULL, 0, s) == -1
    assert g(*args, 4, 8, 256, 128, h.ptr(), h.ptr(), h.ptr(), 2, 3, h.ptr(), 0, s) == -2
    assert g(*args, 4, 8, 256, 128, h.ptr(), h.ptr(), h.ptr(), 0, 4, h.ptr(), 1, s) == -2    # no general-tile flag
    assert g(*args, 4, 8, 256, 64, h.ptr(), h.ptr(), h.ptr(), 0, 4, h.ptr(), 2, s) == -3     # tiled: G >= 128
    assert g(*args, 4, 8, 256, 128, h.ptr(), h.ptr(), h.ptr(), 0, 4, h.ptr(8), 0, s) == -4


def test_tiled_validation(L):
    h = Host()
    b = ctypes.c_int64(-1)
    q = L.apex4_tiled_weights_size
    assert q(8, 256, None) == -1
    assert q(0, 256, ctypes.byref(b)) == -2
    assert q(8, 48, ctypes.byref(b)) == -2 and b.value == -1
    assert q(33, 160, ctypes.byref(b)) == 0 and b.value == 2 * 2 * 2048
    t = L.apex4_tile_weights
    s = NULL
    assert t(NULL, 8, 256, h.ptr(), s) == -1
    assert t(h.ptr(), 8, 256, NULL, s) == -1
    assert t(h.ptr(), 8, 80, h.ptr(), s) == -2
    assert t(h.ptr(), 1 << 20, 1 << 13, h.ptr(), s) == -2                # 4 GiB
    assert t(h.ptr(4), 8, 256, h.ptr(), s) == -4
    g = L.apex4_w4a4_gemm_tiled
    ok = [h.ptr()] * 4
    assert g(NULL, *ok[1:], 4, 8, 256, 128, h.ptr(), NULL, 0, s) == -1
    assert g(*ok, 4, 8, 256, 64, h.ptr(), NULL, 0, s) == -3               # G < 128
    assert g(*ok, 4, 8, 96, 96, h.ptr(), NULL, 0, s) == -3                # G == K < 128
    assert g(*ok, 4, 8, 48, 48, h.ptr(), NULL, 0, s) == -2
    assert g(h.ptr(2), *ok[1:], 4, 8, 8224, 8224, h.ptr(), NULL, 0, s) == -4   # G == K >= 128 accepted
    assert g(*ok, 4, 8, 256, 128, h.ptr(), h.ptr(8), 64, s) == -4         # misaligned workspace
    f = L.apex4_w4a4_linear_tiled
    assert f(NULL, h.ptr(), h.ptr(), 4, 8, 256, 128, h.ptr(), h.ptr(), h.ptr(), s) == -1
    assert f(*[h.ptr()] * 3, 4, 8, 256, 32, h.ptr(), h.ptr(), h.ptr(), s) == -3
    d = L.apex4_w4a4_gemm_debug
    assert d(*ok, 8, 8, 256, 64, h.ptr(), NULL, 0, 0, 8, h.ptr(), 2, s) == -3   # tiled flag with G < 128
    assert d(*ok, 8, 8, 256, 128, h.ptr(), NULL, 0, 0, 8, h.ptr(), 4, s) == -2  # unknown flag


def test_plan_validation(L):
    f = L.apex4_w4a4_gemm_plan
    k, sp = ctypes.c_int(-9), ctypes.c_int(-9)
    assert f(0, 8, 8, 256, 128, 0, None, ctypes.byref(sp)) == -1
    assert f(0, 8, 8, 48, 48, 0, ctypes.byref(k), ctypes.byref(sp)) == -2
    assert f(0, 8, 8, 65568, 65568, 0, ctypes.byref(k), ctypes.byref(sp)) == -3
    assert f(4, 8, 8, 256, 128, 0, ctypes.byref(k), ctypes.byref(sp)) == -2   # unknown entry
    assert f(3, 8, 8, 256, 128, 1, ctypes.byref(k), ctypes.byref(sp)) == -2   # nor for the workspace linear
    assert f(0, 8, 8, 256, 128, 4, ctypes.byref(k), ctypes.byref(sp)) == -2   # unknown flag
    assert f(2, 8, 8, 256, 128, 1, ctypes.byref(k), ctypes.byref(sp)) == -2   # no general tiles for the linear
    assert f(0, 8, 8, 256, 64, 2, ctypes.byref(k), ctypes.byref(sp)) == -3    # tiled needs G >= 128
    assert (k.value, sp.value) == (-9, -9)                                     # nothing written


def test_linear_validation(L):
    h = Host()
    f = L.apex4_w4a4_linear
    s = NULL
    args = lambda **kw: [kw.get(k, h.ptr()) for k in ("x", "wq", "sw")]
    assert f(*args(x=NULL), 4, 8, 256, 128, h.ptr(), h.ptr(), h.ptr(), s) == -1
    assert f(*args(), 4, 8, 256, 128, h.ptr(), NULL, h.ptr(), s) == -1
    assert f(*args(), 4, 8, 200, 128, h.ptr(), h.ptr(), h.ptr(), s) == -2
    assert f(*args(), 4, 8, 384, 96, h.ptr(), h.ptr(), h.ptr(), s) == -3
    assert f(*args(x=h.ptr(2)), 4, 8, 96, 32, h.ptr(), h.ptr(), h.ptr(), s) == -4   # K = 96 accepted
    assert f(*args(x=h.ptr(2)), 4, 8, 256, 128, h.ptr(), h.ptr(), h.ptr(), s) == -4


def test_linear_ws_validation(L):
    h = Host()
    f = L.apex4_w4a4_linear_ws
    s = NULL
    w = lambda **kw: [kw.get(k, h.ptr()) for k in ("x", "w", "sw")]
    tail = lambda ws=None, flags=0: [h.ptr() if ws is None else ws, 1 << 20, flags, s]
    assert f(*w(x=NULL), 4, 8, 256, 128, h.ptr(), h.ptr(), h.ptr(), *tail()) == -1
    assert f(*w(), 4, 8, 256, 128, h.ptr(), NULL, h.ptr(), *tail()) == -1
    assert f(*w(), 4, 8, 200, 128, h.ptr(), h.ptr(), h.ptr(), *tail()) == -2
    assert f(*w(), 4, 8, 384, 96, h.ptr(), h.ptr(), h.ptr(), *tail()) == -3
    assert f(*w(), 4, 8, 256, 128, h.ptr(), h.ptr(), h.ptr(), *tail(flags=1)) == -2    # only the tiled flag
    assert f(*w(), 4, 8, 256, 64, h.ptr(), h.ptr(), h.ptr(), *tail(flags=2)) == -3     # tiled needs G >= 128
    assert f(*w(x=h.ptr(2)), 4, 8, 256, 128, h.ptr(), h.ptr(), h.ptr(), *tail()) == -4
    assert f(*w(), 4, 8, 256, 128, h.ptr(), h.ptr(), h.ptr(), *tail(ws=h.ptr(8))) == -4  # misaligned workspace


def test_fp6_validation(L):
    h = Host()
    f = L.apex4_pack_fp6
    s = NULL
    assert f(NULL, 4, 256, h.ptr(), s) == -1
    assert f(h.ptr(), 4, 256, NULL, s) == -1
    assert f(h.ptr(), -1, 256, h.ptr(), s) == -2
    assert f(h.ptr(), 4, 200, h.ptr(), s) == -2                     # K % 128
    assert f(h.ptr(8), 4, 256, h.ptr(), s) == -4
    g = L.apex4_w4a4_gemm_fp6
    ok = [h.ptr()] * 4
    assert g(NULL, *ok[1:], 4, 8, 256, 128, h.ptr(), s) == -1
    assert g(*ok, 4, 8, 256, 128, NULL, s) == -1
    assert g(*ok, 4, 0, 256, 128, h.ptr(), s) == -2
    assert g(*ok, 4, 8, 320, 128, h.ptr(), s) == -2                # K % 128
    assert g(*ok, 4, 8, 256, 64, h.ptr(), s) == -3                 # G = 128 only
    assert g(*ok, 4, 8, 256, 256, h.ptr(), s) == -3
    assert g(*ok, 1 << 20, 8, 6144, 128, h.ptr(), s) == -2         # A_6 of 4.5 GiB
    assert g(*ok, 4, 1 << 21, 4096, 128, h.ptr(), s) == -2         # W_6 of 6 GiB
    assert g(h.ptr(4), *ok[1:], 4, 8, 256, 128, h.ptr(), s) == -4


def test_workspace_validation(L):
    h = Host()
    q = L.apex4_w4a4_gemm_workspace_size
    b = ctypes.c_int64(-1)
    assert q(4, 8, 256, 128, None) == -1
    assert q(4, 8, 200, 128, ctypes.byref(b)) == -2
    assert q(4, 8, 384, 96, ctypes.byref(b)) == -3
    assert b.value == -1                                           # nothing written on failure
    g = L.apex4_w4a4_gemm_ws
    s = NULL
    ok = [h.ptr()] * 4
    assert g(NULL, *ok[1:], 4, 8, 256, 128, h.ptr(), h.ptr(), 1 << 20, s) == -1
    assert g(*ok, 4, 8, 320, 128, h.ptr(), h.ptr(), 1 << 20, s) == -2
    assert g(*ok, 4, 8, 256, 96, h.ptr(), h.ptr(), 1 << 20, s) == -3
    assert g(*ok, 4, 8, 256, 128, h.ptr(), h.ptr(8), 1 << 20, s) == -4   # misaligned workspace


def test_noalloc_validation(L):
    h = Host()
    g = L.apex4_w4a4_gemm_noalloc
    s = NULL
    ok = [h.ptr()] * 4
    assert g(NULL, *ok[1:], 4, 8, 256, 128, h.ptr(), s) == -1
    assert g(*ok, 4, 8, 256, 128, NULL, s) == -1
    assert g(*ok, 4, 8, 48, 48, h.ptr(), s) == -2
    assert g(*ok, 4, 8, 256, 96, h.ptr(), s) == -3
    assert g(*ok, 4, 8, 256, 128, h.ptr(2), s) == -4


def test_mx_validation(L):
    h = Host()
    q = L.apex4_quantize_mx
    s = NULL
    assert q(NULL, 4, 256, 128, h.ptr(), h.ptr(), s) == -1
    assert q(h.ptr(), 4, 200, 128, h.ptr(), h.ptr(), s) == -2       # K % 128
    assert q(h.ptr(), 4, 256, 96, h.ptr(), h.ptr(), s) == -3        # G not a power of two in 32..1024
    assert q(h.ptr(), 4, 256, 512, h.ptr(), h.ptr(), s) == -3       # G > K
    assert q(h.ptr(), 4, 256, 2048, h.ptr(), h.ptr(), s) == -3
    assert q(h.ptr(), 4, 384, 256, h.ptr(), h.ptr(), s) == -2       # K % G
    assert q(h.ptr(4), 4, 256, 128, h.ptr(), h.ptr(), s) == -4
    g = L.apex4_w4a4_gemm_mx
    ok = [h.ptr()] * 4
    assert g(NULL, *ok[1:], 4, 8, 256, 128, h.ptr(), s) == -1
    assert g(*ok, 4, 8, 256, 128, NULL, s) == -1
    assert g(*ok, 4, 0, 256, 128, h.ptr(), s) == -2
    assert g(*ok, 4, 8, 256, 48, h.ptr(), s) == -3
    assert g(*ok, 1 << 20, 8, 6144, 128, h.ptr(), s) == -2          # A_6 of 4.5 GiB
    assert g(*ok, 4, 8, 256, 128, h.ptr(2), s) == -4
    q = L.apex4_w4a4_gemm_mx_workspace_size
    b = ctypes.c_int64(-1)
    assert q(4, 8, 256, 128, None) == -1
    assert q(4, 8, 200, 128, ctypes.byref(b)) == -2
    assert q(4, 8, 256, 96, ctypes.byref(b)) == -3 and b.value == -1
    w = L.apex4_w4a4_gemm_mx_ws
    assert w(NULL, *ok[1:], 4, 8, 256, 128, h.ptr(), h.ptr(), 1 << 20, s) == -1
    assert w(*ok, 4, 8, 256, 64 * 3, h.ptr(), h.ptr(), 1 << 20, s) == -3
    assert w(*ok, 4, 8, 256, 128, h.ptr(), h.ptr(4), 1 << 20, s) == -4   # misaligned workspace


def test_device_check_without_gpu():
    """Valid arguments on a machine with no gfx950 device: APEX4_ERR_DEVICE, not a crash.
    Run in a child process so the HIP runtime probe stays out of the test process."""
    code = r"""
import ctypes, numpy as np, sys
sys.path.insert(0, %r)
import paper_2606_08761_amd as pk
L = pk.lib()
b = np.zeros(1 << 16, np.uint8); p = ctypes.c_void_p((b.ctypes.data + 255) & ~255)
print(L.apex4_w4a4_gemm(p, p, p, p, 0, 8, 256, 128, p, None))
k = ctypes.c_int(0)
print(L.apex4_w4a4_gemm_plan(0, 8, 8, 96, 32, 0, ctypes.byref(k), ctypes.byref(k)))
print(L.apex4_w4a4_linear_ws(p, p, p, 4, 8, 256, 128, p, p, p, None, 0, 0, None))
""" % ROOT
    try:
        import torch
        if torch.cuda.is_available():
            pytest.skip("a GPU is visible")
    except Exception:
        pass
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip().splitlines()[-3:] == ["-6", "-6", "-6"]


def test_binding_refuses_host_tensors():
    torch = pytest.importorskip("torch")
    import paper_2606_08761_amd as pk
    x = torch.zeros((4, 256), dtype=torch.float16)
    with pytest.raises(TypeError):
        pk.apex4_quantize_act(x, 128)


def test_rho_library_exports_read_probe():
    """The diagnostics library (ρ probes, the counter-calibration copy and the
    streaming-read roofline) exports its entry points and validates arguments
    before touching the GPU."""
    import ctypes
    from paper_2606_08761_amd import rho
    if not os.path.exists(rho.LIB_PATH):
        pytest.skip("librho_apex4.so not built")
    L = rho._lib()
    for name in ("apex4_rho_probe", "apex4_rho_probe_ext", "apex4_rho_probe_issue", "apex4_copy_probe",
                 "apex4_read_probe"):
        assert hasattr(L, name), name
    buf = (ctypes.c_uint8 * 64)()
    base = ctypes.addressof(buf)
    aligned = (base + 15) & ~15
    assert L.apex4_read_probe(None, 16, ctypes.c_void_p(aligned), None) == -1
    assert L.apex4_read_probe(ctypes.c_void_p(aligned), 16, None, None) == -1
    assert L.apex4_read_probe(ctypes.c_void_p(aligned), 15, ctypes.c_void_p(aligned), None) == -1
    assert L.apex4_read_probe(ctypes.c_void_p(aligned + 1), 16, ctypes.c_void_p(aligned), None) == -1
    assert L.apex4_read_probe(ctypes.c_void_p(aligned), 0, ctypes.c_void_p(aligned), None) == 0
