"""rho for the current GPU, measured: the intra-CU ratio of the integer
matrix-core rate to the vector fp32 rate (APEX4 Sec. 2.2, Eqs. T and rho;
Table 1 lists A100 64, RTX 3090 16, A40 16, L40S 8).

Every rate is counted in shader-clock cycles inside the probe kernels
(``rho/rho_probe.hip``), so the clock cancels exactly as in the paper's ratio.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librho_apex4.so")

MFMA_32x32x32_I8_OPS = 2 * 32 * 32 * 32
MFMA_16x16x64_I8_OPS = 2 * 16 * 16 * 64
WAVE = 64
INTERLEAVE_V = (0, 2, 4, 6, 7, 8, 12)
INTERLEAVE_V_2W = (0, 2, 4, 6, 8, 11, 16)


def rho_from_table(int_tops: float, fp32_tflops: float) -> float:
    """rho from a datasheet pair (clock cancels): int-matrix ops / fp32 flops."""
    return int_tops / fp32_tflops


def _lib():
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} missing: run `python -m paper_2606_08761_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    L.apex4_rho_probe.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.c_int]
    L.apex4_rho_probe.restype = ctypes.c_int
    L.apex4_copy_probe.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    L.apex4_copy_probe.restype = ctypes.c_int
    L.apex4_read_probe.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
    L.apex4_read_probe.restype = ctypes.c_int
    L.apex4_rho_probe_ext.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.c_int]
    L.apex4_rho_probe_ext.restype = ctypes.c_int
    L.apex4_rho_probe_issue.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.c_int]
    L.apex4_rho_probe_issue.restype = ctypes.c_int
    return L


def copy(src, dst, stream=None):
    """Device copy of known traffic (the counter calibration reference)."""
    import torch
    if stream is None:
        stream = torch.cuda.current_stream(src.device)
    nbytes = src.numel() * src.element_size()
    rc = _lib().apex4_copy_probe(ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(dst.data_ptr()), nbytes,
                                 ctypes.c_void_p(stream.cuda_stream))
    if rc != 0:
        raise RuntimeError(f"apex4_copy_probe failed: {rc}")


def read(src, sink, stream=None):
    """Plain streaming read of all of `src` (a contiguous device tensor whose
    byte size is a multiple of 16); `sink`: a device tensor of >= 4096 bytes."""
    import torch
    if stream is None:
        stream = torch.cuda.current_stream(src.device)
    if sink.numel() * sink.element_size() < 4096:
        raise ValueError("sink must hold at least 4096 bytes")
    nbytes = src.numel() * src.element_size()
    rc = _lib().apex4_read_probe(ctypes.c_void_p(src.data_ptr()), nbytes, ctypes.c_void_p(sink.data_ptr()),
                                 ctypes.c_void_p(stream.cuda_stream))
    if rc != 0:
        raise RuntimeError(f"apex4_read_probe failed: {rc}")


def measure() -> dict:
    L = _lib()
    out = (ctypes.c_double * 16)()
    rc = L.apex4_rho_probe(out, 16)
    if rc != 0:
        raise RuntimeError(f"apex4_rho_probe failed: {rc}")
    o = list(out)
    mfma_ops_clk_simd = MFMA_32x32x32_I8_OPS / o[0]
    fma_flops_clk_simd = 2 * WAVE / o[2]            # one FMA = 2 flops per lane (one wave per SIMD)
    cvt_ops_clk_simd = 2 * WAVE / o[3]              # two converts per measured pair
    iss = (ctypes.c_double * 9)()
    if L.apex4_rho_probe_issue(iss, 9) != 0:
        raise RuntimeError("apex4_rho_probe_issue failed")
    i9 = list(iss)
    fma_sustained_clk_simd = 2 * WAVE / min(i9[0], i9[1])   # several waves per SIMD
    res = {
        "cycles_per_mfma_i32_32x32x32_i8": o[0],
        "cycles_per_mfma_i32_16x16x64_i8": o[1],
        "cycles_per_v_fma_f32": o[2],
        "cycles_per_cvt_pair": o[3],
        "int8_mfma_ops_per_clk_per_cu": 4 * mfma_ops_clk_simd,
        "int8_mfma16_ops_per_clk_per_cu": 4 * MFMA_16x16x64_I8_OPS / o[1],
        "fp32_fma_flops_per_clk_per_cu": 4 * fma_flops_clk_simd,
        "cvt_ops_per_clk_per_cu": 4 * cvt_ops_clk_simd,
        "rho_measured": mfma_ops_clk_simd / fma_sustained_clk_simd,
        "rho_measured_one_wave_per_simd": mfma_ops_clk_simd / fma_flops_clk_simd,
        "cycles_per_v_fma_f32_per_simd_2_waves": i9[0],
        "cycles_per_v_fma_f32_per_simd_4_waves": i9[1],
        "fp32_fma_flops_per_clk_per_cu_sustained": 4 * fma_sustained_clk_simd,
        "mfma_cycles_per_simd_2_waves_v_fma_interleaved": {str(v): i9[2 + i] for i, v in enumerate(INTERLEAVE_V_2W)},
        "rho_datasheet_packed_fp32": rho_from_table(5033.2, 157.3),
        "rho_datasheet_unpacked_fp32": rho_from_table(5033.2, 78.6),
        "mfma_cycles_with_v_fma_interleaved": {str(v): o[4 + i] for i, v in enumerate(INTERLEAVE_V)},
        "split_waves_mfma_cycles": o[11],
        "split_waves_fma_cycles": o[12],
        "lds_read_b128_bytes_per_clk_per_cu": o[13],
        "shader_clock_mhz": o[14],
        "cus": int(o[15]),
    }
    ext = (ctypes.c_double * 5)()
    if L.apex4_rho_probe_ext(ext, 5) == 0:
        e = list(ext)
        res.update({
            "mfma_cycles_1_dependent_chain": e[0],
            "mfma_cycles_2_chains": e[1],
            "mfma_cycles_1_chain_per_wave_2_waves_per_simd": e[2],
            "lds_read_b128_bytes_per_clk_per_cu_4w16": e[3],
            "lds_read_b128_bytes_per_clk_per_cu_8w16": e[4],
        })
    return res


if __name__ == "__main__":
    import json
    print(json.dumps(measure(), indent=1))
