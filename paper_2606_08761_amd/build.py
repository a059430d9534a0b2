"""Build the HIP library ``libapex4.so`` for gfx950, in-tree.

    python -m paper_2606_08761_amd.build

All HIP sources under ``csrc/`` are compiled by hipcc for gfx950 only.
Packed-FP32 instructions are disabled (``-packed-fp32-ops``); binary32
division and square root stay correctly rounded (the quantizer relies on it).
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libapex4.so")
RHO_SRC = os.path.join(HERE, "rho", "rho_probe.hip")
RHO_LIB = os.path.join(HERE, "librho_apex4.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

HIP_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-fno-fast-math",
    "-ffp-contract=fast",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wno-unused-command-line-argument",
]


def sources() -> list[str]:
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _hipcc(srcs: list[str], out: str, verbose: bool) -> None:
    cmd = [HIPCC, *HIP_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", *srcs, "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature and says so; that is harmless
    err = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip())
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
    if verbose and err:
        print(err, file=sys.stderr)
    os.replace(out + ".tmp", out)


def build(verbose: bool = False) -> str:
    """Build libapex4.so (the product) and librho_apex4.so (the rho probes)."""
    _hipcc(sources(), LIB, verbose)
    _hipcc([RHO_SRC], RHO_LIB, verbose)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
