"""MI355X-native W4A4 group-quantized GEMM (the hot path of APEX4, arXiv 2606.08761).

Thin Python binding over the C ABI in ``include/apex4.h`` (``libapex4.so``).
The functions carry the C names and only marshal arguments: torch supplies
device memory and the stream, every step of the computation runs in the HIP
kernels.  There is no fallback: if the library is missing or the device is
not gfx950 the call raises.

    A_q, s_a = apex4_quantize_act(x, G)                 # x: [M, K] float16 on cuda
    Y = apex4_w4a4_gemm(A_q, s_a, W_q, s_w, G)          # Y: [M, N] float16
    P = apex4_w4a4_gemm_groupsums(A_q, W_q, G, m0, mr)  # int32 [mr, N, K/G]
    Y = apex4_w4a4_linear(x, W_q, s_w, G)               # quantize + GEMM
    lin = W4A4Linear(w, G); y = lin(x)                  # drop-in layer (weights quantized once)
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libapex4.so")

APEX4_OK = 0
STATUS = {0: "APEX4_OK", -1: "APEX4_ERR_NULL", -2: "APEX4_ERR_SHAPE", -3: "APEX4_ERR_GROUP",
          -4: "APEX4_ERR_ALIGN", -5: "APEX4_ERR_LAUNCH", -6: "APEX4_ERR_DEVICE", -7: "APEX4_ERR_WORKSPACE"}
APEX4_DEBUG_GENERAL_TILES = 1
APEX4_DEBUG_W_TILED = 2
APEX4_NOALLOC_SCRATCH_BYTES = 32 << 20
ENTRY = {"gemm": 0, "gemm_ws": 1, "linear": 2, "linear_ws": 3}
KERNELS = {0: None, 1: "gemv", 2: "fused", 3: "decode", 4: "tile64", 5: "tile128", 6: "pingpong",
           7: "decode_split"}

EXPORTED = ("apex4_quantize_act", "apex4_w4a4_gemm", "apex4_w4a4_gemm_groupsums", "apex4_w4a4_gemm_debug",
            "apex4_w4a4_gemm_plan", "apex4_w4a4_linear", "apex4_w4a4_linear_debug", "apex4_pack_fp6",
            "apex4_w4a4_gemm_fp6", "apex4_w4a4_gemm_workspace_size", "apex4_w4a4_gemm_ws",
            "apex4_w4a4_gemm_noalloc", "apex4_quantize_mx", "apex4_w4a4_gemm_mx",
            "apex4_w4a4_gemm_mx_workspace_size", "apex4_w4a4_gemm_mx_ws", "apex4_status_string",
            "apex4_version", "apex4_tiled_weights_size", "apex4_tile_weights", "apex4_w4a4_gemm_tiled",
            "apex4_w4a4_linear_tiled", "apex4_w4a4_linear_ws")

_lib = None


class Apex4Error(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn}: {msg}")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded ``libapex4.so`` with its argument types declared."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2606_08761_amd.build` (no fallback path exists)")
    L = ctypes.CDLL(LIB_PATH)
    P, I = ctypes.c_void_p, ctypes.c_int64
    L.apex4_quantize_act.argtypes = [P, I, I, I, P, P, P]
    L.apex4_w4a4_gemm.argtypes = [P, P, P, P, I, I, I, I, P, P]
    L.apex4_w4a4_gemm_groupsums.argtypes = [P, P, I, I, I, I, I, I, P, P]
    L.apex4_w4a4_gemm_debug.argtypes = [P, P, P, P, I, I, I, I, P, P, I, I, I, P, ctypes.c_int, P]
    L.apex4_w4a4_gemm_plan.argtypes = [ctypes.c_int, I, I, I, I, ctypes.c_int, P, P]
    L.apex4_w4a4_linear.argtypes = [P, P, P, I, I, I, I, P, P, P, P]
    L.apex4_w4a4_linear_debug.argtypes = [P, P, P, I, I, I, I, P, P, P, I, I, P, ctypes.c_int, P]
    L.apex4_tiled_weights_size.argtypes = [I, I, P]
    L.apex4_tile_weights.argtypes = [P, I, I, P, P]
    L.apex4_w4a4_gemm_tiled.argtypes = [P, P, P, P, I, I, I, I, P, P, I, P]
    L.apex4_w4a4_linear_tiled.argtypes = [P, P, P, I, I, I, I, P, P, P, P]
    L.apex4_w4a4_linear_ws.argtypes = [P, P, P, I, I, I, I, P, P, P, P, I, ctypes.c_int, P]
    L.apex4_pack_fp6.argtypes = [P, I, I, P, P]
    L.apex4_w4a4_gemm_workspace_size.argtypes = [I, I, I, I, P]
    L.apex4_quantize_mx.argtypes = [P, I, I, I, P, P, P]
    L.apex4_w4a4_gemm_mx.argtypes = [P, P, P, P, I, I, I, I, P, P]
    L.apex4_w4a4_gemm_mx_workspace_size.argtypes = [I, I, I, I, P]
    L.apex4_w4a4_gemm_mx_ws.argtypes = [P, P, P, P, I, I, I, I, P, P, I, P]
    L.apex4_w4a4_gemm_ws.argtypes = [P, P, P, P, I, I, I, I, P, P, I, P]
    L.apex4_w4a4_gemm_noalloc.argtypes = [P, P, P, P, I, I, I, I, P, P]
    L.apex4_w4a4_gemm_fp6.argtypes = [P, P, P, P, I, I, I, I, P, P]
    for f in ("apex4_quantize_act", "apex4_w4a4_gemm", "apex4_w4a4_gemm_groupsums", "apex4_w4a4_gemm_debug",
              "apex4_w4a4_gemm_plan", "apex4_w4a4_linear", "apex4_w4a4_linear_debug", "apex4_pack_fp6",
              "apex4_w4a4_gemm_fp6", "apex4_w4a4_gemm_workspace_size", "apex4_w4a4_gemm_ws",
              "apex4_w4a4_gemm_noalloc", "apex4_quantize_mx", "apex4_w4a4_gemm_mx",
              "apex4_w4a4_gemm_mx_workspace_size", "apex4_w4a4_gemm_mx_ws", "apex4_tiled_weights_size",
              "apex4_tile_weights", "apex4_w4a4_gemm_tiled", "apex4_w4a4_linear_tiled", "apex4_w4a4_linear_ws"):
        getattr(L, f).restype = ctypes.c_int
    L.apex4_status_string.argtypes = [ctypes.c_int]
    L.apex4_status_string.restype = ctypes.c_char_p
    L.apex4_version.argtypes = []
    L.apex4_version.restype = ctypes.c_int
    _lib = L
    return L


def _check(fn: str, rc: int):
    if rc != APEX4_OK:
        raise Apex4Error(fn, rc, lib().apex4_status_string(rc).decode())


def _stream(t, stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream(t.device)
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t, dtype, name):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def apex4_quantize_act(x, G: int, A_q=None, s_a=None, stream=None):
    """SymQuant (b=4) of a [M, K] float16 tensor in groups of G along K.

    Returns (A_q uint8 [M, K/2], s_a float16 [M, K/G])."""
    import torch
    M, K = x.shape
    if A_q is None:
        A_q = torch.empty((M, K // 2), dtype=torch.uint8, device=x.device)
    if s_a is None:
        s_a = torch.empty((M, max(K // G, 1)), dtype=torch.float16, device=x.device)
    rc = lib().apex4_quantize_act(_dev(x, torch.float16, "x"), M, K, G, _dev(A_q, torch.uint8, "A_q"),
                                  _dev(s_a, torch.float16, "s_a"), _stream(x, stream))
    _check("apex4_quantize_act", rc)
    return A_q, s_a


def apex4_w4a4_gemm(A_q, s_a, W_q, s_w, G: int, Y=None, stream=None):
    """Y[M, N] = sum_g s_a[:, g] s_w[:, g]^T (.) (A_q,g W_q,g^T), float16 output."""
    import torch
    M, K2 = A_q.shape
    N = W_q.shape[0]
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float16, device=A_q.device)
    rc = lib().apex4_w4a4_gemm(_dev(A_q, torch.uint8, "A_q"), _dev(s_a, torch.float16, "s_a"),
                               _dev(W_q, torch.uint8, "W_q"), _dev(s_w, torch.float16, "s_w"),
                               M, N, 2 * K2, G, _dev(Y, torch.float16, "Y"), _stream(A_q, stream))
    _check("apex4_w4a4_gemm", rc)
    return Y


def apex4_w4a4_gemm_workspace_size(M: int, N: int, K: int, G: int) -> int:
    """Bytes of workspace apex4_w4a4_gemm_ws needs for this shape on the current device (0: none)."""
    b = ctypes.c_int64(0)
    _check("apex4_w4a4_gemm_workspace_size", lib().apex4_w4a4_gemm_workspace_size(M, N, K, G, ctypes.byref(b)))
    return int(b.value)


def apex4_w4a4_gemm_ws(A_q, s_a, W_q, s_w, G: int, workspace=None, Y=None, stream=None):
    """apex4_w4a4_gemm split over K when its tiles leave CUs idle; workspace is a
    uint8 device tensor of at least apex4_w4a4_gemm_workspace_size bytes (made
    here when None)."""
    import torch
    M, K2 = A_q.shape
    N, K = W_q.shape[0], 2 * K2
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float16, device=A_q.device)
    if workspace is None:
        need = apex4_w4a4_gemm_workspace_size(M, N, K, G)
        workspace = torch.empty((max(need, 16),), dtype=torch.uint8, device=A_q.device)
    rc = lib().apex4_w4a4_gemm_ws(_dev(A_q, torch.uint8, "A_q"), _dev(s_a, torch.float16, "s_a"),
                                  _dev(W_q, torch.uint8, "W_q"), _dev(s_w, torch.float16, "s_w"),
                                  M, N, K, G, _dev(Y, torch.float16, "Y"), _dev(workspace, torch.uint8, "workspace"),
                                  workspace.numel(), _stream(A_q, stream))
    _check("apex4_w4a4_gemm_ws", rc)
    return Y


def apex4_w4a4_gemm_noalloc(A_q, s_a, W_q, s_w, G: int, Y=None, stream=None):
    """apex4_w4a4_gemm_ws with the library's static per-device scratch in place
    of a workspace: the C call allocates nothing (Y is made here when None)."""
    import torch
    M, K2 = A_q.shape
    N = W_q.shape[0]
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float16, device=A_q.device)
    rc = lib().apex4_w4a4_gemm_noalloc(_dev(A_q, torch.uint8, "A_q"), _dev(s_a, torch.float16, "s_a"),
                                       _dev(W_q, torch.uint8, "W_q"), _dev(s_w, torch.float16, "s_w"),
                                       M, N, 2 * K2, G, _dev(Y, torch.float16, "Y"), _stream(A_q, stream))
    _check("apex4_w4a4_gemm_noalloc", rc)
    return Y


def apex4_w4a4_gemm_groupsums(A_q, W_q, G: int, m0: int = 0, mr: int | None = None, P=None, stream=None):
    """Exact int32 group sums P[i, n, g] for rows m0 .. m0+mr-1 (debug dump)."""
    import torch
    M, K2 = A_q.shape
    N, K = W_q.shape[0], 2 * K2
    if mr is None:
        mr = M - m0
    if P is None:
        P = torch.empty((mr, N, max(K // G, 1)), dtype=torch.int32, device=A_q.device)
    rc = lib().apex4_w4a4_gemm_groupsums(_dev(A_q, torch.uint8, "A_q"), _dev(W_q, torch.uint8, "W_q"),
                                         M, N, K, G, m0, mr, _dev(P, torch.int32, "P"),
                                         _stream(A_q, stream))
    _check("apex4_w4a4_gemm_groupsums", rc)
    return P


def _window(M, N, K, G, m0, mr, P, device):
    import torch
    if mr is None:
        mr = M - m0
    if P is None:
        P = torch.empty((mr, N, max(K // G, 1)), dtype=torch.int32, device=device)
    return mr, P


def apex4_w4a4_gemm_debug(A_q, s_a, W_q, s_w, G: int, m0: int = 0, mr: int | None = None, workspace=None,
                          flags: int = 0, Y=None, P=None, stream=None):
    """Y of apex4_w4a4_gemm (workspace None) or apex4_w4a4_gemm_ws (workspace a
    uint8 device tensor) and, from the same launches, the exact int32 group
    sums P[i, n, g] of rows m0 .. m0+mr-1.  Returns (Y, P).  With
    flags & APEX4_DEBUG_W_TILED, W_q is tiled (N from s_w)."""
    import torch
    M, K2 = A_q.shape
    N, K = s_w.shape[0], 2 * K2
    mr, P = _window(M, N, K, G, m0, mr, P, A_q.device)
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float16, device=A_q.device)
    ws = ctypes.c_void_p(0) if workspace is None else _dev(workspace, torch.uint8, "workspace")
    rc = lib().apex4_w4a4_gemm_debug(_dev(A_q, torch.uint8, "A_q"), _dev(s_a, torch.float16, "s_a"),
                                     _dev(W_q, torch.uint8, "W_q"), _dev(s_w, torch.float16, "s_w"),
                                     M, N, K, G, _dev(Y, torch.float16, "Y"), ws,
                                     0 if workspace is None else workspace.numel(), m0, mr,
                                     _dev(P, torch.int32, "P"), flags, _stream(A_q, stream))
    _check("apex4_w4a4_gemm_debug", rc)
    return Y, P


def apex4_w4a4_linear(x, W_q, s_w, G: int, Y=None, A_q_work=None, s_a_work=None, stream=None):
    """Quantize x (SymQuant) then the W4A4 GEMM, both enqueued on one stream."""
    import torch
    M, K = x.shape
    N = W_q.shape[0]
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float16, device=x.device)
    if A_q_work is None:
        A_q_work = torch.empty((M, K // 2), dtype=torch.uint8, device=x.device)
    if s_a_work is None:
        s_a_work = torch.empty((M, max(K // G, 1)), dtype=torch.float16, device=x.device)
    rc = lib().apex4_w4a4_linear(_dev(x, torch.float16, "x"), _dev(W_q, torch.uint8, "W_q"),
                                 _dev(s_w, torch.float16, "s_w"), M, N, K, G,
                                 _dev(Y, torch.float16, "Y"), _dev(A_q_work, torch.uint8, "A_q_work"),
                                 _dev(s_a_work, torch.float16, "s_a_work"), _stream(x, stream))
    _check("apex4_w4a4_linear", rc)
    return Y


def apex4_w4a4_gemm_plan(entry: str, M: int, N: int, K: int, G: int, flags: int = 0):
    """(kernel name, splits) that the entry point ("gemm", "gemm_ws", "linear"
    or "linear_ws") runs for this shape on the current device."""
    k, s = ctypes.c_int(0), ctypes.c_int(0)
    _check("apex4_w4a4_gemm_plan", lib().apex4_w4a4_gemm_plan(ENTRY[entry], M, N, K, G, flags, ctypes.byref(k),
                                                              ctypes.byref(s)))
    return KERNELS[k.value], int(s.value)


def apex4_w4a4_linear_debug(x, W_q, s_w, G: int, m0: int = 0, mr: int | None = None, Y=None, A_q_work=None,
                            s_a_work=None, P=None, flags: int = 0, stream=None):
    """apex4_w4a4_linear (or, with flags=APEX4_DEBUG_W_TILED, apex4_w4a4_linear_tiled)
    plus the exact int32 group sums of rows m0 .. m0+mr-1 from the same
    kernels.  Returns (Y, A_q_work, s_a_work, P)."""
    import torch
    M, K = x.shape
    N = s_w.shape[0]
    mr, P = _window(M, N, K, G, m0, mr, P, x.device)
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float16, device=x.device)
    if A_q_work is None:
        A_q_work = torch.empty((M, K // 2), dtype=torch.uint8, device=x.device)
    if s_a_work is None:
        s_a_work = torch.empty((M, max(K // G, 1)), dtype=torch.float16, device=x.device)
    rc = lib().apex4_w4a4_linear_debug(_dev(x, torch.float16, "x"), _dev(W_q, torch.uint8, "W_q"),
                                       _dev(s_w, torch.float16, "s_w"), M, N, K, G, _dev(Y, torch.float16, "Y"),
                                       _dev(A_q_work, torch.uint8, "A_q_work"), _dev(s_a_work, torch.float16, "s_a_work"),
                                       m0, mr, _dev(P, torch.int32, "P"), flags, _stream(x, stream))
    _check("apex4_w4a4_linear_debug", rc)
    return Y, A_q_work, s_a_work, P


def apex4_tiled_weights_size(N: int, K: int) -> int:
    """Bytes of the tiled layout of an [N, K/2] packed weight matrix."""
    b = ctypes.c_int64(0)
    _check("apex4_tiled_weights_size", lib().apex4_tiled_weights_size(N, K, ctypes.byref(b)))
    return int(b.value)


def apex4_tile_weights(W_q, W_t=None, stream=None):
    """Packed weight codes uint8 [N, K/2] -> the tiled layout, a flat uint8 tensor
    (offline, once per weight matrix)."""
    import torch
    N, K2 = W_q.shape
    if W_t is None:
        W_t = torch.empty((apex4_tiled_weights_size(N, 2 * K2),), dtype=torch.uint8, device=W_q.device)
    rc = lib().apex4_tile_weights(_dev(W_q, torch.uint8, "W_q"), N, 2 * K2, _dev(W_t, torch.uint8, "W_t"),
                                  _stream(W_q, stream))
    _check("apex4_tile_weights", rc)
    return W_t


def apex4_w4a4_gemm_tiled(A_q, s_a, W_t, s_w, G: int, workspace=None, Y=None, stream=None):
    """apex4_w4a4_gemm on tiled weights (N from s_w); with a workspace tensor, the
    apex4_w4a4_gemm_ws kernel choice (split over K where it applies)."""
    import torch
    M, K2 = A_q.shape
    N = s_w.shape[0]
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float16, device=A_q.device)
    ws = ctypes.c_void_p(0) if workspace is None else _dev(workspace, torch.uint8, "workspace")
    rc = lib().apex4_w4a4_gemm_tiled(_dev(A_q, torch.uint8, "A_q"), _dev(s_a, torch.float16, "s_a"),
                                     _dev(W_t, torch.uint8, "W_t"), _dev(s_w, torch.float16, "s_w"), M, N, 2 * K2, G,
                                     _dev(Y, torch.float16, "Y"), ws, 0 if workspace is None else workspace.numel(),
                                     _stream(A_q, stream))
    _check("apex4_w4a4_gemm_tiled", rc)
    return Y


def apex4_w4a4_linear_tiled(x, W_t, s_w, G: int, Y=None, A_q_work=None, s_a_work=None, stream=None):
    """apex4_w4a4_linear on tiled weights (N from s_w)."""
    import torch
    M, K = x.shape
    N = s_w.shape[0]
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float16, device=x.device)
    if A_q_work is None:
        A_q_work = torch.empty((M, K // 2), dtype=torch.uint8, device=x.device)
    if s_a_work is None:
        s_a_work = torch.empty((M, max(K // G, 1)), dtype=torch.float16, device=x.device)
    rc = lib().apex4_w4a4_linear_tiled(_dev(x, torch.float16, "x"), _dev(W_t, torch.uint8, "W_t"),
                                       _dev(s_w, torch.float16, "s_w"), M, N, K, G, _dev(Y, torch.float16, "Y"),
                                       _dev(A_q_work, torch.uint8, "A_q_work"), _dev(s_a_work, torch.float16, "s_a_work"),
                                       _stream(x, stream))
    _check("apex4_w4a4_linear_tiled", rc)
    return Y


def apex4_w4a4_linear_ws(x, W, s_w, G: int, workspace=None, tiled: bool = False, Y=None, A_q_work=None,
                         s_a_work=None, stream=None, make_workspace: bool = True):
    """apex4_w4a4_linear (tiled=True: apex4_w4a4_linear_tiled) with the GEMM
    split over K, or in its stream-K form, where apex4_w4a4_gemm_ws would be;
    workspace is a uint8 device tensor of at least
    apex4_w4a4_gemm_workspace_size bytes.  When it is None: with
    make_workspace, one is made here if the shape needs one; without, none is
    passed (for callers that know the shape needs none).  N from s_w."""
    import torch
    M, K = x.shape
    N = s_w.shape[0]
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float16, device=x.device)
    if A_q_work is None:
        A_q_work = torch.empty((M, K // 2), dtype=torch.uint8, device=x.device)
    if s_a_work is None:
        s_a_work = torch.empty((M, max(K // G, 1)), dtype=torch.float16, device=x.device)
    if workspace is None and M and make_workspace:
        need = apex4_w4a4_gemm_workspace_size(M, N, K, G)
        if need:
            workspace = torch.empty((need,), dtype=torch.uint8, device=x.device)
    ws = ctypes.c_void_p(0) if workspace is None else _dev(workspace, torch.uint8, "workspace")
    rc = lib().apex4_w4a4_linear_ws(_dev(x, torch.float16, "x"), _dev(W, torch.uint8, "W"),
                                    _dev(s_w, torch.float16, "s_w"), M, N, K, G, _dev(Y, torch.float16, "Y"),
                                    _dev(A_q_work, torch.uint8, "A_q_work"), _dev(s_a_work, torch.float16, "s_a_work"),
                                    ws, 0 if workspace is None else workspace.numel(),
                                    APEX4_DEBUG_W_TILED if tiled else 0, _stream(x, stream))
    _check("apex4_w4a4_linear_ws", rc)
    return Y


def apex4_pack_fp6(q4, q6=None, stream=None):
    """Packed 4-bit codes uint8 [rows, K/2] -> FP6 e3m2 codes uint8 [rows, 3K/4]."""
    import torch
    rows, K2 = q4.shape
    K = 2 * K2
    if q6 is None:
        q6 = torch.empty((rows, 3 * K // 4), dtype=torch.uint8, device=q4.device)
    rc = lib().apex4_pack_fp6(_dev(q4, torch.uint8, "q4"), rows, K, _dev(q6, torch.uint8, "q6"), _stream(q4, stream))
    _check("apex4_pack_fp6", rc)
    return q6


def apex4_w4a4_gemm_fp6(A_6, s_a, W_6, s_w, G: int, Y=None, stream=None):
    """apex4_w4a4_gemm on FP6 containers (A_6 [M, 3K/4], W_6 [N, 3K/4]); G = 128."""
    import torch
    M, K34 = A_6.shape
    N = W_6.shape[0]
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float16, device=A_6.device)
    rc = lib().apex4_w4a4_gemm_fp6(_dev(A_6, torch.uint8, "A_6"), _dev(s_a, torch.float16, "s_a"),
                                   _dev(W_6, torch.uint8, "W_6"), _dev(s_w, torch.float16, "s_w"),
                                   M, N, 4 * K34 // 3, G, _dev(Y, torch.float16, "Y"), _stream(A_6, stream))
    _check("apex4_w4a4_gemm_fp6", rc)
    return Y


def apex4_quantize_mx(x, G: int, Q6=None, e=None, stream=None):
    """MX variant quantizer: x [M, K] float16 -> (FP6 codes uint8 [M, 3K/4], E8M0 scales uint8 [M, K/G])."""
    import torch
    M, K = x.shape
    if Q6 is None:
        Q6 = torch.empty((M, 3 * K // 4), dtype=torch.uint8, device=x.device)
    if e is None:
        e = torch.empty((M, K // G), dtype=torch.uint8, device=x.device)
    rc = lib().apex4_quantize_mx(_dev(x, torch.float16, "x"), M, K, G, _dev(Q6, torch.uint8, "Q6"),
                                 _dev(e, torch.uint8, "e"), _stream(x, stream))
    _check("apex4_quantize_mx", rc)
    return Q6, e


def apex4_w4a4_gemm_mx(A_6, e_a, W_6, e_w, G: int, Y=None, stream=None):
    """MX variant GEMM: power-of-two group scales applied inside the FP6 MFMA."""
    import torch
    M, K34 = A_6.shape
    N = W_6.shape[0]
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float16, device=A_6.device)
    rc = lib().apex4_w4a4_gemm_mx(_dev(A_6, torch.uint8, "A_6"), _dev(e_a, torch.uint8, "e_a"),
                                  _dev(W_6, torch.uint8, "W_6"), _dev(e_w, torch.uint8, "e_w"),
                                  M, N, 4 * K34 // 3, G, _dev(Y, torch.float16, "Y"), _stream(A_6, stream))
    _check("apex4_w4a4_gemm_mx", rc)
    return Y


def apex4_w4a4_gemm_mx_workspace_size(M: int, N: int, K: int, G: int) -> int:
    """Bytes of workspace apex4_w4a4_gemm_mx_ws needs for this shape on the current device (0: none)."""
    b = ctypes.c_int64(0)
    _check("apex4_w4a4_gemm_mx_workspace_size", lib().apex4_w4a4_gemm_mx_workspace_size(M, N, K, G, ctypes.byref(b)))
    return int(b.value)


def apex4_w4a4_gemm_mx_ws(A_6, e_a, W_6, e_w, G: int, workspace=None, Y=None, stream=None):
    """apex4_w4a4_gemm_mx split over K when its tiles leave CUs idle (workspace made here when None)."""
    import torch
    M, K34 = A_6.shape
    N, K = W_6.shape[0], 4 * K34 // 3
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float16, device=A_6.device)
    if workspace is None:
        need = apex4_w4a4_gemm_mx_workspace_size(M, N, K, G)
        workspace = torch.empty((max(need, 16),), dtype=torch.uint8, device=A_6.device)
    rc = lib().apex4_w4a4_gemm_mx_ws(_dev(A_6, torch.uint8, "A_6"), _dev(e_a, torch.uint8, "e_a"),
                                     _dev(W_6, torch.uint8, "W_6"), _dev(e_w, torch.uint8, "e_w"), M, N, K, G,
                                     _dev(Y, torch.float16, "Y"), _dev(workspace, torch.uint8, "workspace"),
                                     workspace.numel(), _stream(A_6, stream))
    _check("apex4_w4a4_gemm_mx_ws", rc)
    return Y


def apex4_version() -> int:
    return int(lib().apex4_version())


class W4A4Linear:
    """Drop-in W4A4 linear layer over the C ABI (APEX4 Sec. 3.2.1, Sec. 4.4):
    the fp16 weight [N, K] is quantized once with SymQuant (b=4, group G, the
    same formula as the activations) and packed offline, and every forward
    quantizes the fp16 activations on the fly and runs the W4A4 GEMM.

        lin = W4A4Linear(weight_fp16_cuda, G=128)
        y = lin(x)             # x [..., K] float16 on the same device -> [..., N]

    layout="auto" keeps the weights in the tiled layout (apex4_tile_weights)
    where it applies (G >= 128, fp16 scales) and row-major otherwise; "rows"
    or "tiled" force one.  Only that copy is kept (W_q for rows, W_t for
    tiled).

    scales="mx" selects the MX variant instead: power-of-two group scales
    applied inside the FP6 matrix instruction (apex4_quantize_mx +
    apex4_w4a4_gemm_mx_ws; G in 32..1024) -- not the paper's fp16 scales.

    Work buffers (quantized activations, split-K workspace) are cached per
    (row count, stream), so forwards on different streams never share them;
    calls with the same row count on one stream reuse them in stream order.
    Bias and other dtypes are not supported: the paper's layers are bias-free
    fp16 linears."""

    MAX_CACHED = 8

    def __init__(self, weight, G: int = 128, scales: str = "fp16", layout: str = "auto"):
        import torch
        if weight.dim() != 2:
            raise ValueError("weight must be [N, K]")
        if scales not in ("fp16", "mx"):
            raise ValueError("scales must be 'fp16' or 'mx'")
        if layout not in ("auto", "rows", "tiled"):
            raise ValueError("layout must be 'auto', 'rows' or 'tiled'")
        self.N, self.K = weight.shape
        self.G = self.K if G in (0, None) else int(G)
        self.mx = scales == "mx"
        tiled_ok = not self.mx and self.G >= 128
        if layout == "tiled" and not tiled_ok:
            raise ValueError("the tiled layout needs fp16 scales and G >= 128")
        self.tiled = tiled_ok if layout == "auto" else layout == "tiled"
        quant = apex4_quantize_mx if self.mx else apex4_quantize_act
        W_q, self.s_w = quant(weight.contiguous(), self.G)
        self.W_q, self.W_t = (None, apex4_tile_weights(W_q)) if self.tiled else (W_q, None)
        del W_q
        self._work = {}
        self.device = weight.device
        self._torch = torch

    def _buffers(self, M, stream):
        key = (M, stream.cuda_stream)
        buf = self._work.pop(key, None)
        if buf is None:
            torch = self._torch
            size = apex4_w4a4_gemm_mx_workspace_size if self.mx else apex4_w4a4_gemm_workspace_size
            need = size(M, self.N, self.K, self.G) if M else 0
            codes = (M, 3 * self.K // 4) if self.mx else (M, self.K // 2)
            sdt = torch.uint8 if self.mx else torch.float16
            buf = (torch.empty(codes, dtype=torch.uint8, device=self.device),
                   torch.empty((M, max(self.K // self.G, 1)), dtype=sdt, device=self.device),
                   torch.empty((need,), dtype=torch.uint8, device=self.device) if need else None)
            while len(self._work) >= self.MAX_CACHED:
                self._work.pop(next(iter(self._work)))
        self._work[key] = buf  # most recently used last
        return buf

    def __call__(self, x, stream=None):
        lead = x.shape[:-1]
        if x.shape[-1] != self.K:
            raise ValueError(f"expected last dimension {self.K}, got {x.shape[-1]}")
        x2 = x.reshape(-1, self.K).contiguous()
        M = x2.shape[0]
        if stream is None:
            stream = self._torch.cuda.current_stream(x2.device)
        Aq, sa, ws = self._buffers(M, stream)
        if self.mx:
            apex4_quantize_mx(x2, self.G, Aq, sa, stream=stream)
            if ws is None:
                Y = apex4_w4a4_gemm_mx(Aq, sa, self.W_q, self.s_w, self.G, stream=stream)
            else:
                Y = apex4_w4a4_gemm_mx_ws(Aq, sa, self.W_q, self.s_w, self.G, ws, stream=stream)
        else:
            # one C call: the quantizer, then the GEMM (split over K or stream-K
            # where the cached workspace exists; fused for one row where it pays)
            W = self.W_t if self.tiled else self.W_q
            Y = apex4_w4a4_linear_ws(x2, W, self.s_w, self.G, workspace=ws, tiled=self.tiled, A_q_work=Aq,
                                     s_a_work=sa, stream=stream, make_workspace=False)
        return Y.reshape(*lead, self.N)
