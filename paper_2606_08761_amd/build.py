"""Build the HIP library ``libapex4.so`` for gfx950, in-tree.

    python -m paper_2606_08761_amd.build

All HIP sources under ``csrc/`` are compiled by hipcc for gfx950 only.
Packed-FP32 instructions are disabled (``-packed-fp32-ops``); binary32
division and square root stay correctly rounded (the quantizer relies on it).
"""
from __future__ import annotations

import glob
import json
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libapex4.so")
# per-kernel registers and scratch of the last build (the compiler's resource remarks)
RESOURCES = os.path.join(HERE, "kernel_resources.json")
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


def _resources(stderr: str) -> dict:
    """{kernel: {"vgpr": n, "agpr": n, "scratch": bytes per lane, "occupancy": waves per SIMD}}
    from -Rpass-analysis=kernel-resource-usage remarks."""
    res, name = {}, None
    keys = {"VGPRs": "vgpr", "AGPRs": "agpr", "ScratchSize [bytes/lane]": "scratch", "Occupancy [waves/SIMD]": "occupancy"}
    for line in stderr.splitlines():
        m = re.search(r"remark: .*?Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            res.setdefault(name, {})
            continue
        m = re.search(r"remark: .*?\s(VGPRs|AGPRs|ScratchSize \[bytes/lane\]|Occupancy \[waves/SIMD\]): (\d+)", line)
        if m and name:
            res[name][keys[m.group(1)]] = int(m.group(2))
    return res


def _hipcc(srcs: list[str], out: str, verbose: bool, resources: str | None = None) -> None:
    extra = ["-Rpass-analysis=kernel-resource-usage"] if resources else []
    cmd = [HIPCC, *HIP_FLAGS, *extra, f"-I{INCLUDE}", f"-I{CSRC}", *srcs, "-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if resources and res.returncode == 0:
        with open(resources, "w") as f:
            json.dump(_resources(res.stderr), f, indent=0, sort_keys=True)
    # hipcc's host pass does not know the packed-fp32 feature and says so; that
    # is harmless; the resource remarks went to the file above
    err = "\n".join(l for l in res.stderr.splitlines()
                    if "packed-fp32-ops" not in l and "kernel-resource-usage" not in l and l.strip()
                    and not re.match(r"^\s*\d*\s*\|", l))
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
    if verbose and err:
        print(err, file=sys.stderr)
    os.replace(out + ".tmp", out)


def build(verbose: bool = False) -> str:
    """Build libapex4.so (the product) and librho_apex4.so (the rho probes)."""
    _hipcc(sources(), LIB, verbose, RESOURCES)
    _hipcc([RHO_SRC], RHO_LIB, verbose)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
