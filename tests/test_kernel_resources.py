"""Register use of the built GEMM kernels (no GPU needed).

The build records the compiler's resource remarks for every kernel of
libapex4.so (paper_2606_08761_amd/kernel_resources.json).  A production kernel
that spills to scratch runs several times slower while its results stay right
(a 6x slowdown of the G = 32 tile kernel once passed every parity test), so
the spill-free state is checked here.  Exempt: the debug instantiations (group
sum dumps) and the partial-last-stage forms (K % 128 != 0), which serve tests
and rare shapes.
"""
import json
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
RES = os.path.join(ROOT, "paper_2606_08761_amd", "kernel_resources.json")

# kernel name -> positions of its (DUMP, TAIL) template arguments (None: absent)
FLAGS = {
    "w4a4_gemm_kernel": (9, 10),
    "w4a4_gemm_pp_kernel": (0, None),
    "w4a4_decode_kernel": (3, 4),
    "w4a4_gemv_kernel": (2, None),
    "w4a4_gemv_tiled_kernel": (2, None),
}


@pytest.fixture(scope="module")
def kernels():
    if not os.path.exists(RES):
        from paper_2606_08761_amd import build
        build.build()
    with open(RES) as f:
        res = json.load(f)
    names = list(res)
    out = subprocess.run(["c++filt"], input="\n".join(names), capture_output=True, text=True, check=True)
    return {d: res[m] for m, d in zip(names, out.stdout.splitlines())}


def _template_args(demangled):
    m = re.search(r"::(\w+)<([^()]*)>\(", demangled)
    if not m:
        m2 = re.search(r"::(\w+)\(", demangled)
        return (m2.group(1) if m2 else demangled), []
    return m.group(1), [a.strip() for a in m.group(2).split(",")]


def test_every_kernel_reported(kernels):
    names = {_template_args(d)[0] for d in kernels}
    for k in ("w4a4_gemm_kernel", "w4a4_gemm_pp_kernel", "w4a4_decode_kernel", "w4a4_gemv_kernel",
              "w4a4_gemv_tiled_kernel", "tile_weights_kernel"):
        assert k in names, k
    assert all("scratch" in v and "vgpr" in v for v in kernels.values())


def test_production_kernels_do_not_spill(kernels):
    spills = []
    for d, r in kernels.items():
        name, args = _template_args(d)
        dump_at, tail_at = FLAGS.get(name, (None, None))
        flag = lambda at: at is not None and at < len(args) and args[at] == "true"
        exempt = flag(dump_at) or flag(tail_at)
        if r["scratch"] and not exempt:
            spills.append(f"{name}<{', '.join(args)}>: {r['scratch']} bytes/lane, {r['vgpr']} VGPRs")
    assert not spills, "production kernels spill:\n" + "\n".join(spills)
