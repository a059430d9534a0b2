"""Shared helpers of the GPU parity tests (host side only)."""
from __future__ import annotations

import sys

import numpy as np

# Output tolerance for the binary16 GEMM result against the oracle's binary64 y
# (before its rounding):  |Y - y| <= 2e-3 |y| + 1e-2 RMS_row(y).
# The binary16 rounding alone contributes <= 2^-11 |y| ~ 4.9e-4 |y|; the binary32
# accumulation of K/G scaled group sums adds ~ sqrt(K/G) * 2^-24 * max|term|,
# far below the RMS term.
TOL_REL = 2e-3
TOL_RMS = 1e-2


def log(*a):
    print("[parity]", *a, flush=True)
    sys.stdout.flush()


def dev(a: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t) -> np.ndarray:
    return t.cpu().numpy()


def check_tolerance(Y16: np.ndarray, y: np.ndarray, what: str = ""):
    Y = Y16.astype(np.float64)
    rms = np.sqrt(np.mean(y * y, axis=1, keepdims=True))
    err = np.abs(Y - y)
    bound = TOL_REL * np.abs(y) + TOL_RMS * rms
    bad = err > bound
    if bad.any():
        i, j = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} elements out of tolerance; first at ({i},{j}): "
                             f"Y={Y[i, j]!r} y={y[i, j]!r} bound={bound[i, j]!r}")
    assert np.isfinite(Y).all()


def sample_rows(M: int, seed: int = 0, n_random: int = 6, tile: int = 128) -> np.ndarray:
    """Row 0, the last row, rows on both sides of tile boundaries, and random rows."""
    rows = {0, M - 1}
    for b in (tile, 2 * tile, M // 2):
        for r in (b - 1, b):
            if 0 <= r < M:
                rows.add(r)
    rng = np.random.default_rng(seed)
    rows.update(int(r) for r in rng.integers(0, M, size=n_random))
    return np.array(sorted(rows), dtype=np.int64)
