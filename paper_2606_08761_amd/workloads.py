"""Seeded synthetic inputs with the shapes and value distributions of the
paper's GEMM workloads.

This module holds no arithmetic of the method: it only draws random numbers
and converts them to the storage types the boundary takes.  Both the HIP path
and the CPU oracle consume exactly the bytes produced here.

Workloads (the paper measures N = K = 8192 GEMM sweeps and the linear layers of
Llama-2/Qwen2.5; Sec. 2.1 Fig. 1, Sec. 5.3, Sec. 5.5 Fig. ratio).  No dataset is
used: random integers and Gaussian activations/weights stand in for them.

  tiny        M=64,  N=K=1024,  G=128   random codes + scales
  paper       M=2048, N=K=8192, G=128   random codes + scales (the headline GEMM)
  llama70b    (N,K) in {(10240,8192) qkv, (8192,8192) o, (57344,8192) gate+up,
              (8192,28672) down} x M in {16,256,4096}, G=128, activations
              N(0,1) with 1% outlier channels x20, weights N(0,0.02)
  gsweep      M=4096, N=K=8192, G in {128,256,512,8192}, as llama70b
  decode      M in {1,8,32}, (N,K) in {(8192,8192),(28672,8192)}, G=128,
              as llama70b, quantize + GEMM timed together

Seeds: numpy SeedSequence([0xA9E4, workload_id, tensor_id]).
"""
from __future__ import annotations

import numpy as np

SEED_ROOT = 0xA9E4

WORKLOAD_IDS = {"tiny": 0, "paper": 1, "llama70b": 2, "gsweep": 3, "decode": 4}

LLAMA70B_LINEARS = {
    "qkv": (10240, 8192),
    "o_proj": (8192, 8192),
    "gate_up": (57344, 8192),
    "down": (8192, 28672),
}


def rng_for(workload: str | int, tensor_id: int, extra: int = 0) -> np.random.Generator:
    wid = WORKLOAD_IDS[workload] if isinstance(workload, str) else int(workload)
    return np.random.default_rng(np.random.SeedSequence([SEED_ROOT, wid, tensor_id, extra]))


def random_codes(rng: np.random.Generator, rows: int, K: int) -> np.ndarray:
    """Packed signed 4-bit codes, i.i.d. uniform over [-8, 7].

    A uniformly random byte is exactly two independent uniform nibbles, so the
    packed array is drawn directly: [rows, K/2] uint8, low nibble = even k."""
    return rng.integers(0, 256, size=(rows, K // 2), dtype=np.uint8)


def random_scales(rng: np.random.Generator, rows: int, ngroups: int,
                  lo: float = 0.005, hi: float = 0.02) -> np.ndarray:
    """binary16 scales drawn uniform in [lo, hi]."""
    return rng.uniform(lo, hi, size=(rows, ngroups)).astype(np.float16)


def activations(rng: np.random.Generator, M: int, K: int, outlier_frac: float = 0.01,
                outlier_gain: float = 20.0, outlier_cols: np.ndarray | None = None) -> np.ndarray:
    """binary16 activations ~ N(0,1) with a fixed set of outlier channels.

    The same 1% of the K columns is scaled by 20 in every row (channel-wise
    outliers, as the paper describes for LLM activations in Sec. 3.1)."""
    x = rng.standard_normal((M, K), dtype=np.float32)
    if outlier_cols is None:
        outlier_cols = outlier_channels(K, outlier_frac)
    x[:, outlier_cols] *= outlier_gain
    return x.astype(np.float16)


def outlier_channels(K: int, frac: float = 0.01) -> np.ndarray:
    r = np.random.default_rng(np.random.SeedSequence([SEED_ROOT, 99, K]))
    n = max(1, int(round(K * frac)))
    return np.sort(r.choice(K, size=n, replace=False))


def weights(rng: np.random.Generator, N: int, K: int, std: float = 0.02) -> np.ndarray:
    """binary16 weights ~ N(0, std), stored [N, K] (nn.Linear convention)."""
    return (rng.standard_normal((N, K), dtype=np.float32) * np.float32(std)).astype(np.float16)


def codes_workload(workload: str, M: int, N: int, K: int, G: int):
    """Random packed codes and scales for a GEMM (the tiny and paper workloads)."""
    r = rng_for(workload, 0, M * 1_000_003 + N * 1009 + K + G)
    Aq = random_codes(r, M, K)
    Wq = random_codes(r, N, K)
    sa = random_scales(r, M, K // G)
    sw = random_scales(r, N, K // G)
    return Aq, sa, Wq, sw


def float_workload(workload: str, M: int, N: int, K: int, tensor_tag: int = 0):
    """binary16 activations and weights (the llama70b, gsweep and decode workloads)."""
    r = rng_for(workload, 1 + tensor_tag, M * 1_000_003 + N * 1009 + K)
    x = activations(r, M, K)
    w = weights(r, N, K)
    return x, w
