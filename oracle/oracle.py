"""ctypes front end of the CPU oracle (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  The product library never does.

Every function takes and returns numpy arrays:
  * binary16 data are passed as ``numpy.float16`` arrays (their bit patterns
    are what the C code reads);
  * packed codes are ``uint8`` arrays of shape [rows, K/2], low nibble = even k.

Paper: APEX4 (arXiv 2606.08761), Sec. 3.2.1 -- Eq. (SymQuant) for
``quantize`` and Eq. (group_decomposition) for ``groupsums``/``gemm_rows``.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle_apex4.so")

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from . import build as _b  # noqa: F401  (package-relative when imported as oracle.oracle)
        _b.build()
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    I = ctypes.c_int64
    lib.apex4o_f16_to_f64.argtypes = [ctypes.c_uint16]
    lib.apex4o_f16_to_f64.restype = ctypes.c_double
    lib.apex4o_f64_to_f16.argtypes = [ctypes.c_double]
    lib.apex4o_f64_to_f16.restype = ctypes.c_uint16
    lib.apex4o_f16_to_f64_n.argtypes = [P, I, P]
    lib.apex4o_f16_to_f64_n.restype = None
    lib.apex4o_f64_to_f16_n.argtypes = [P, I, P]
    lib.apex4o_f64_to_f16_n.restype = None
    lib.apex4o_quantize.argtypes = [P, I, I, I, P, P]
    lib.apex4o_quantize.restype = ctypes.c_int
    lib.apex4o_groupsums.argtypes = [P, P, I, I, I, I, I, I, P]
    lib.apex4o_groupsums.restype = ctypes.c_int
    lib.apex4o_gemm_rows.argtypes = [P, P, P, P, I, I, I, I, P, I, P]
    lib.apex4o_gemm_rows.restype = ctypes.c_int
    lib.apex4o_num_threads.argtypes = []
    lib.apex4o_num_threads.restype = ctypes.c_int
    lib.apex4o_set_num_threads.argtypes = [ctypes.c_int]
    lib.apex4o_set_num_threads.restype = None
    _lib = lib
    return lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def f16_to_f64(h: np.ndarray) -> np.ndarray:
    """binary16 -> binary64 (exact).  ``h`` is float16 or uint16 bit patterns."""
    h = _c(np.asarray(h).view(np.uint16) if np.asarray(h).dtype == np.float16 else h, np.uint16)
    out = np.empty(h.shape, np.float64)
    _load().apex4o_f16_to_f64_n(_ptr(h), h.size, _ptr(out))
    return out


def f64_to_f16(x: np.ndarray) -> np.ndarray:
    """binary64 -> binary16, round to nearest even.  Returns float16."""
    x = _c(x, np.float64)
    out = np.empty(x.shape, np.uint16)
    _load().apex4o_f64_to_f16_n(_ptr(x), x.size, _ptr(out))
    return out.view(np.float16)


def quantize(x: np.ndarray, G: int):
    """SymQuant of a [R, K] float16 matrix in groups of G along K.

    Returns (q_packed uint8 [R, K/2], scales float16 [R, K/G])."""
    x = _c(x, np.float16)
    R, K = x.shape
    q = np.empty((R, K // 2), np.uint8)
    s = np.empty((R, K // G), np.float16)
    rc = _load().apex4o_quantize(_ptr(x), R, K, G, _ptr(q), _ptr(s))
    if rc != 0:
        raise ValueError(f"oracle quantize: bad shape R={R} K={K} G={G}")
    return q, s


def groupsums(Aq: np.ndarray, Wq: np.ndarray, K: int, G: int, m0: int = 0, mr: int | None = None):
    """Exact int64 group sums P[i, n, g] for rows m0 .. m0+mr-1."""
    Aq = _c(Aq, np.uint8)
    Wq = _c(Wq, np.uint8)
    M, N = Aq.shape[0], Wq.shape[0]
    if mr is None:
        mr = M - m0
    P = np.empty((mr, N, K // G), np.int64)
    rc = _load().apex4o_groupsums(_ptr(Aq), _ptr(Wq), M, N, K, G, m0, mr, _ptr(P))
    if rc != 0:
        raise ValueError("oracle groupsums: bad arguments")
    return P


def gemm_rows(Aq, sa, Wq, sw, K: int, G: int, rows=None):
    """binary64 y[i, n] = sum_g s_a s_w P for the listed rows (all rows if None)."""
    Aq = _c(Aq, np.uint8)
    Wq = _c(Wq, np.uint8)
    sa = _c(sa, np.float16)
    sw = _c(sw, np.float16)
    M, N = Aq.shape[0], Wq.shape[0]
    if rows is None:
        rows = np.arange(M, dtype=np.int64)
    rows = _c(rows, np.int64)
    y = np.empty((rows.size, N), np.float64)
    rc = _load().apex4o_gemm_rows(_ptr(Aq), _ptr(sa), _ptr(Wq), _ptr(sw), M, N, K, G,
                                  _ptr(rows), rows.size, _ptr(y))
    if rc != 0:
        raise ValueError("oracle gemm_rows: bad arguments")
    return y


def gemm_f16(Aq, sa, Wq, sw, K: int, G: int, rows=None):
    """Y = binary16(y), one rounding from binary64."""
    return f64_to_f16(gemm_rows(Aq, sa, Wq, sw, K, G, rows))


def num_threads() -> int:
    return int(_load().apex4o_num_threads())


def set_num_threads(n: int) -> None:
    """Threads for the following oracle calls (timing only; results do not depend on it)."""
    _load().apex4o_set_num_threads(int(n))
