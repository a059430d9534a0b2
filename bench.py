#!/usr/bin/env python3
"""Benchmark of the W4A4 group-quantized linear on one MI355X.

    python bench.py [--gpus 1] [--steps 50] [--warmup 10]

One step is one pass of the whole hot path over one batch: the per-token,
per-group SymQuant of fp16 activations x [M, K] (apex4_quantize_act) followed
by the W4A4 group GEMM against offline-quantized weights (apex4_w4a4_gemm),
both enqueued on one stream -- apex4_w4a4_linear.  Workload: the paper's
compute-bound GEMM shape M=2048, N=K=8192, G=128 (APEX4 Fig. 1 / Sec. 5.3 use
N=K=8192), synthetic seeded data, inputs resident in HBM before timing.
The inputs are rotated over several copies (> 2x the 256 MB Infinity Cache).

Printed JSON line (rank 0): the metric is TOPS = 2 M N K / t_step; it also
carries the GEMM kernel's roofline (live HIP-event timing of the GEMM launches
inside the timed region), the fp16 hipBLASLt GEMM of the same shape, and the
CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

INT8_PEAK_TOPS = 5033.2     # MI355X dense INT8 MFMA: 256 CU x 8192 op/clk x 2.4 GHz
FP16_PEAK_TFLOPS = 2516.6   # MI355X dense FP16 MFMA
HBM_PEAK_GBS = 8000.0

M, N, K, G = 2048, 8192, 8192, 128
ROTATE_BYTES = 512 << 20


class TimingEvent:
    """A HIP event used only to take GPU timestamps between kernels.

    Created with hipEventDisableSystemFence (0x20000000): recording it issues
    no system-scope release, i.e. no L2 write-back and invalidation at every
    mark.  torch's events (default flags) do issue one; between back-to-back
    kernels on MI355X each such mark costs about 3 us of step time, 1.5 us
    without the fence.  The timed region still ends with a full device
    synchronization, so the wall clock covers all of the work.  The calls go
    to the HIP runtime already mapped into the process (the one torch and
    libapex4 use)."""

    FLAGS = 0x20000000
    _hip = None

    @classmethod
    def runtime(cls):
        if cls._hip is None:
            import ctypes
            path = "libamdhip64.so.7"
            with open("/proc/self/maps") as f:
                for line in f:
                    if "libamdhip64" in line:
                        path = line.split()[-1]
                        break
            cls._hip = ctypes.CDLL(path)
        return cls._hip

    def __init__(self):
        import ctypes
        self._c = ctypes
        self.h = ctypes.c_void_p()
        rc = self.runtime().hipEventCreateWithFlags(ctypes.byref(self.h), ctypes.c_uint(self.FLAGS))
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")

    def record(self, stream):
        rc = self.runtime().hipEventRecord(self.h, self._c.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def elapsed_time(self, end) -> float:
        """Milliseconds from this event to `end` (both complete)."""
        ms = self._c.c_float()
        rc = self.runtime().hipEventElapsedTime(self._c.byref(ms), self.h, end.h)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return ms.value

    def destroy(self):
        if self.h:
            self.runtime().hipEventDestroy(self.h)
            self.h = self._c.c_void_p()


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-decode", action="store_true", help="skip the decode-size linears")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="target oracle sample duration")
    p.add_argument("--mode", choices=("bench", "counters", "rho", "summarize", "gsweep", "power", "layers", "variants",
                                      "decode_counters", "decode_split", "decode_sq"),
                   default="bench",
                   help="counters: 3 GEMM launches + 3 copies of 256 MiB, for rocprofv3 --pmc; "
                        "rho: the intra-CU throughput probes; "
                        "summarize: turn rocprofv3 CSV output into the profiles/ summaries")
    p.add_argument("--fetch-csv", help="summarize: counter_collection.csv of the FETCH_SIZE pass")
    p.add_argument("--write-csv", help="summarize: counter_collection.csv of the WRITE_SIZE pass")
    p.add_argument("--stats-csv", help="summarize: kernel_stats.csv of the --kernel-trace --stats run")
    p.add_argument("--commands", help="summarize: text file with the exact commands that made the CSVs")
    p.add_argument("--bench-log", help="summarize: output of the traced bench run (its JSON line)")
    p.add_argument("--gsweep-trace", help="summarize: kernel_trace.csv of the --kernel-trace run of --mode gsweep")
    p.add_argument("--rho-json", help="summarize: output of --mode rho (written to profiles/rho_probes.md)")
    p.add_argument("--rho-command", default="python3 bench.py --mode rho", help="summarize: the command that made --rho-json")
    p.add_argument("--gsweep-pmc", help="summarize: counter_collection.csv of the SQ counter pass over --mode gsweep")
    p.add_argument("--sq-csv", nargs="*", help="summarize: counter_collection.csv files of SQ counter passes over --mode counters")
    p.add_argument("--sq-commands", help="summarize: text file with the commands that made --sq-csv")
    p.add_argument("--variants-sq-csv", nargs="*", help="summarize: counter_collection.csv files of SQ passes over --mode variants")
    p.add_argument("--variants-commands", help="summarize: text file with the commands that made --variants-sq-csv")
    p.add_argument("--power-log", help="summarize: output of --mode power (written to profiles/power_clock_paper_shape.md)")
    p.add_argument("--power-command", default="python3 bench.py --mode power", help="summarize: the command that made --power-log")
    p.add_argument("--layers-log", help="summarize: output of --mode layers (written to profiles/layer_sweep_llama2_70b.md)")
    p.add_argument("--decode-fetch-csv", help="summarize: counter_collection.csv of the FETCH_SIZE pass over --mode decode_counters")
    p.add_argument("--decode-write-csv", help="summarize: counter_collection.csv of the WRITE_SIZE pass over --mode decode_counters")
    p.add_argument("--decode-trace-csv", help="summarize: kernel_trace.csv of the --kernel-trace run of --mode decode_counters")
    p.add_argument("--decode-log", help="summarize: output of --mode decode_counters (its JSON line)")
    p.add_argument("--decode-commands", help="summarize: text file with the commands that made the --decode-* files")
    p.add_argument("--decode-sq-csv", nargs="*",
                   help="summarize: counter_collection.csv files of SQ passes over --mode decode_sq")
    p.add_argument("--decode-sq-commands", help="summarize: text file with the commands that made --decode-sq-csv")
    p.add_argument("--layers-command", default="python3 bench.py --mode layers", help="summarize: the command that made --layers-log")
    return p.parse_args()


def is_tiled_gemm(name: str) -> bool:
    """Kernel-trace / counter rows of the tiled GEMM (both G = 128 ping-pong and the general kernel)."""
    return "w4a4_gemm_kernel" in name or "w4a4_gemm_pp_kernel" in name


def traffic_from_profile():
    """HBM bytes per GEMM launch from the committed counter summary, if it was
    taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "gemm_w4a4_paper_traffic.json")
    src = os.path.join(ROOT, "paper_2606_08761_amd", "csrc", "gemm_w4a4.hip")
    try:
        with open(path) as f:
            prof = json.load(f)
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
        if prof.get("kernel_source_sha256") != sha:
            return None
        return float(prof["hbm_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def host_cpu_model() -> str:
    """The host CPU's model name (from /proc/cpuinfo), or "unknown"."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(target_s: float, threads: int = 0):
    """The oracle (quantize the sampled activation rows + binary64 GEMM rows)
    timed on this host for a bounded row sample; TOPS scaled to 2 * rows * N * K.
    threads > 0 pins the oracle's OpenMP thread count (default: all)."""
    from oracle import oracle as O
    from paper_2606_08761_amd import workloads as wl

    x, w = wl.float_workload("paper", M, N, K)
    Wq, sw = O.quantize(w, G)                       # weights are quantized offline
    if threads > 0:
        O.set_num_threads(threads)
    rows = 2
    while True:
        t0 = time.perf_counter()
        Aq, sa = O.quantize(x[:rows], G)
        O.gemm_rows(Aq, sa, Wq, sw, K, G)
        dt = time.perf_counter() - t0
        if dt >= target_s / 2 or rows >= M:
            break
        rows = min(M, max(rows * 2, int(rows * target_s / max(dt, 1e-3) / 2)))
    reps = 1
    while dt * reps < target_s and reps < 8:       # repeat the whole-M sample up to the target
        t0 = time.perf_counter()
        Aq, sa = O.quantize(x[:rows], G)
        O.gemm_rows(Aq, sa, Wq, sw, K, G)
        dt = (dt * reps + time.perf_counter() - t0) / (reps + 1)
        reps += 1
    tops = 2.0 * rows * N * K / dt / 1e12
    return {"value": tops, "unit": "TOPS", "cores": O.num_threads(), "kind": "oracle", "cpu": host_cpu_model(),
            "sample": f"{rows} of {M} rows of the M={M} N={N} K={K} G={G} linear "
                      f"(quantize rows + int64/fp64 GEMM rows), mean of {reps} run(s) of {dt:.1f} s"}


def summarize_mode(args):
    """profiles/gemm_w4a4_paper_traffic.json and profiles/gemm_w4a4_paper_shape.md from
    rocprofv3 output.  FETCH_SIZE / WRITE_SIZE (KiB per dispatch) are scaled by
    what the same counter reads for the 256 MiB reference copy."""
    import csv
    import statistics

    def per_kernel(path, counter):
        vals = {}
        for r in csv.DictReader(open(path)):
            if r.get("Counter_Name") != counter:
                continue
            vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return vals

    def pick(vals, key):
        xs = [v for k, vs in vals.items() if key in k for v in vs]
        return statistics.mean(xs) if xs else None

    if args.decode_fetch_csv:
        summarize_decode_traffic(args)
    if not (args.fetch_csv and args.write_csv and args.stats_csv):
        if args.layers_log:
            summarize_layers(args.layers_log, args.layers_command)
        if args.sq_csv:
            summarize_sq(args.sq_csv, open(args.sq_commands).read().strip() if args.sq_commands else "")
        if args.variants_sq_csv:
            summarize_sq_variants(args.variants_sq_csv,
                                  open(args.variants_commands).read().strip() if args.variants_commands else "")
        if args.power_log:
            summarize_power(args.power_log, args.power_command)
        if args.rho_json:
            summarize_rho(args.rho_json, args.rho_command)
        if args.decode_sq_csv:
            summarize_decode_sq(args.decode_sq_csv,
                                open(args.decode_sq_commands).read().strip() if args.decode_sq_commands else "")
        return
    copy_kib = (256 << 20) / 1024.0
    fetch = per_kernel(args.fetch_csv, "FETCH_SIZE")
    write = per_kernel(args.write_csv, "WRITE_SIZE")
    f_copy, w_copy = pick(fetch, "copy_kernel"), pick(write, "copy_kernel")
    f_gemm, w_gemm = pick(fetch, "w4a4_gemm_pp_kernel"), pick(write, "w4a4_gemm_pp_kernel")
    f_scale, w_scale = copy_kib / f_copy, copy_kib / w_copy
    read_b = f_gemm * f_scale * 1024.0
    write_b = w_gemm * w_scale * 1024.0
    alg = M * K // 2 + N * K // 2 + 2 * (M + N) * (K // G) + 2 * M * N
    src = os.path.join(ROOT, "paper_2606_08761_amd", "csrc", "gemm_w4a4.hip")
    stats = list(csv.DictReader(open(args.stats_csv)))
    cmds = open(args.commands).read().strip() if args.commands else ""
    prof = {
        "kernel": "w4a4_gemm_pp_kernel (G=128, 128 x 256 tiles, ping-pong)",
        "workload": f"M={M} N={N} K={K} G={G}",
        "kernel_source_sha256": hashlib.sha256(open(src, "rb").read()).hexdigest(),
        "fetch_kib_per_dispatch": f_gemm, "write_kib_per_dispatch": w_gemm,
        "copy_fetch_kib": f_copy, "copy_write_kib": w_copy, "copy_bytes": 256 << 20,
        "fetch_scale": f_scale, "write_scale": w_scale,
        "hbm_read_bytes_per_launch": read_b, "hbm_write_bytes_per_launch": write_b,
        "hbm_bytes_per_launch": read_b + write_b,
        "algorithmic_bytes_per_launch": alg,
        "commands": cmds,
    }
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", "gemm_w4a4_paper_traffic.json"), "w") as f:
        json.dump(prof, f, indent=1)
    lines = ["# W4A4 GEMM, M=2048 N=K=8192 G=128: rocprofv3 summary", "",
             "Commands (run from the repository root on one MI355X):", "", "```", cmds, "```", "",
             "## Kernel trace (`--kernel-trace --stats`, bench.py default workload)", "",
             "| kernel | calls | avg us | min us | max us |", "|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"]))[:12]:
        name = r["Name"]
        m = re.search(r"(\w+_kernel(?:<[^()]*>)?)", name)
        short = (m.group(1) if m else name.split("(")[0])[:80]
        lines.append(f"| `{short}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} |")
    lines += ["", "## HBM traffic of the GEMM (`--pmc FETCH_SIZE`, then `--pmc WRITE_SIZE`, `bench.py --mode counters`)", "",
              f"* reference copy of 256 MiB: FETCH_SIZE {f_copy:.0f} KiB (scale {f_scale:.3f}), "
              f"WRITE_SIZE {w_copy:.0f} KiB (scale {w_scale:.3f})",
              f"* GEMM per dispatch: FETCH_SIZE {f_gemm:.0f} KiB -> {read_b / 1e6:.1f} MB read; "
              f"WRITE_SIZE {w_gemm:.0f} KiB -> {write_b / 1e6:.1f} MB written",
              f"* algorithmic bytes per launch: {alg / 1e6:.1f} MB; measured / algorithmic = "
              f"{(read_b + write_b) / alg:.2f}",
              f"* kernel source sha256: `{prof['kernel_source_sha256']}`"]
    if args.bench_log:
        line = [l for l in open(args.bench_log) if l.startswith("{")][-1]
        b = json.loads(line)
        lines += ["", "## Per-workload timing of the traced bench run (HIP events in bench.py, same process)", "",
                  f"* quantizer, x[{M},{K}] G={G}: {b['quant_us']:.1f} us ({b['quant_hbm_gbs']:.0f} GB/s of "
                  f"{2.5 * M * K + 2 * M * K / G:.3g} algorithmic bytes)",
                  f"* W4A4 GEMM {M}x{N}x{K} G={G}: {b['gemm_us']:.1f} us ({b['gemm_tops']:.0f} TOPS); "
                  f"fp16 GEMM (hipBLASLt) {b['fp16_gemm_us']:.1f} us",
                  "", "Decode linears: eager = one Python call per launch (partly launch-bound at these sizes); "
                  "graph = the same calls replayed from a captured graph (GPU time, used for GB/s).", "",
                  "Linear = apex4_w4a4_linear from fp16 x (one fused kernel at M=1 where it pays, quantizer + GEMM otherwise); "
                  "quantize then GEMM = the two entry points called in turn.", "",
                  "Weights in the tiled layout; the row-major column runs the same GEMM on row-major weights.", "",
                  "Plain read = a streaming read kernel (librho_apex4 apex4_read_probe) over the same rotated "
                  "weight copies, graph-timed the same way: the rate any kernel that reads those bytes once "
                  "reaches at that size; GEMM / read = read time / GEMM time.", "",
                  "| decode M | N | K | kernel | linear us (eager / graph) | quantize then GEMM us (graph) | "
                  "GEMM us (eager / graph) | GEMM HBM GB/s (fraction of 8 TB/s) | plain read us (fraction of 8 TB/s) | "
                  "GEMM / read | row-major GEMM us (graph) | fp16 GEMM us (eager) | linear speedup vs fp16 (eager / graph) |",
                  "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
        for d in b.get("decode", []):
            lines.append(f"| {d['M']} | {d['N']} | {d['K']} | {d.get('kernel')} | {d['linear_us']} / {d.get('linear_graph_us')} | "
                         f"{d.get('quant_then_gemm_graph_us')} | {d['gemm_us']} / {d.get('gemm_graph_us')} | "
                         f"{d['gemm_hbm_gbs']} ({d['gemm_hbm_frac']}) | {d.get('read_graph_us')} ({d.get('read_hbm_frac')}) | "
                         f"{d.get('gemm_rate_vs_read')} | {d.get('row_major_gemm_graph_us')} | "
                         f"{d['fp16_gemm_us']} | {d['speedup_linear_vs_fp16']} / {d.get('speedup_linear_graph_vs_fp16')} |")
    with open(os.path.join(ROOT, "profiles", "gemm_w4a4_paper_shape.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    if args.gsweep_trace and args.gsweep_pmc:
        summarize_gsweep(args.gsweep_trace, args.gsweep_pmc, cmds)
    if args.rho_json:
        summarize_rho(args.rho_json, args.rho_command)
    if args.sq_csv:
        summarize_sq(args.sq_csv, open(args.sq_commands).read().strip() if args.sq_commands else "")
    if args.power_log:
        summarize_power(args.power_log, args.power_command)
    print(json.dumps(prof, indent=1))


# Llama-2-70B decoder-layer linears (hidden 8192, 64 query heads and 8 KV heads of
# 128, FFN 28672): (name, N, K, G) with G = 0 meaning per-channel (G = K).  "g128"
# is the paper's uniform configuration; "mix" its mixed granularity (Sec. 3.2.2):
# G = 32 for the value and down projections, per-channel for every other linear.
LAYER_CONFIGS = {
    "g128": [("qkv", 10240, 8192, 128), ("o", 8192, 8192, 128), ("gate_up", 57344, 8192, 128),
             ("down", 8192, 28672, 128)],
    "mix": [("qk", 9216, 8192, 0), ("v", 1024, 8192, 32), ("o", 8192, 8192, 0), ("gate_up", 57344, 8192, 0),
            ("down", 8192, 28672, 32)],
}
LAYER_M = (16, 256, 4096)
# The MX variant (power-of-two group scales inside the FP6 MFMA; not the
# paper's fp16 scales) on the same linears, uniformly at G = 32 and G = 128.
MX_LAYER_CONFIGS = {
    "mx_g32": [(n, N_, K_, 32) for n, N_, K_, _ in LAYER_CONFIGS["g128"]],
    "mx_g128": [(n, N_, K_, 128) for n, N_, K_, _ in LAYER_CONFIGS["g128"]],
}


def decode_split_mode(reps: int = 40, rounds: int = 6):
    """The few-row GEMM with and without a workspace (round robin against the
    stream-K form where the plan takes it), over N x K x G x M; graph replay of
    `reps` calls, the two forms alternated `rounds` times (median), weights
    rotated past the Infinity Cache.  Writes profiles/decode_stream_k.md."""
    import statistics
    import torch
    import paper_2606_08761_amd as pk
    from paper_2606_08761_amd import workloads as wl
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)

    def capture(fn):
        side = torch.cuda.Stream(dev)
        side.wait_stream(stream)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            for i in range(reps):
                fn(i)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        return g

    def once(g):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3

    rows = []
    for G in (32, 128):
        for K in (8192, 28672):
            for N in (64, 256, 1024, 2048, 4096, 8192, 10240):
                for M in (4, 16):
                    tiled = G >= 128
                    kern, _ = pk.apex4_w4a4_gemm_plan("gemm_ws", M, N, K, G, pk.APEX4_DEBUG_W_TILED if tiled else 0)
                    need = pk.apex4_w4a4_gemm_workspace_size(M, N, K, G)
                    r = wl.rng_for("decode", 7, M * 100003 + N * 7 + K + G)
                    Wq = torch.from_numpy(wl.random_codes(r, N, K)).to(dev)
                    W = pk.apex4_tile_weights(Wq) if tiled else Wq
                    sw = torch.from_numpy(wl.random_scales(r, N, K // G)).to(dev)
                    R = max(2, -(-ROTATE_BYTES // W.numel()))
                    wset = [W.clone() for _ in range(R)]
                    x = torch.from_numpy(wl.activations(r, M, K)).to(dev)
                    Aq, sa = pk.apex4_quantize_act(x, G)
                    work = torch.empty((max(need, 16),), dtype=torch.uint8, device=dev)
                    Y0 = torch.empty((M, N), dtype=torch.float16, device=dev)
                    Y1 = torch.empty_like(Y0)
                    if tiled:
                        def f0(i):
                            pk.apex4_w4a4_gemm_tiled(Aq, sa, wset[i % R], sw, G, None, Y0)

                        def f1(i):
                            pk.apex4_w4a4_gemm_tiled(Aq, sa, wset[i % R], sw, G, work, Y1)
                    else:
                        def f0(i):
                            pk.apex4_w4a4_gemm(Aq, sa, wset[i % R], sw, G, Y0)

                        def f1(i):
                            pk.apex4_w4a4_gemm_ws(Aq, sa, wset[i % R], sw, G, work, Y1)
                    g0, g1 = capture(f0), capture(f1)
                    t0, t1 = [], []
                    for _ in range(rounds):
                        t0.append(once(g0))
                        t1.append(once(g1))
                    del g0, g1, wset, W, Wq
                    a, b = statistics.median(t0), statistics.median(t1)
                    row = {"mode": "decode_split", "M": M, "N": N, "K": K, "G": G, "plan_ws": kern,
                           "workspace_bytes": need, "round_robin_us": round(a, 2), "workspace_us": round(b, 2),
                           "ratio": round(b / a, 3)}
                    rows.append(row)
                    print(json.dumps(row), flush=True)
    lines = ["# Few-row GEMM: round robin against the stream-K form", "",
             "Command (run from the repository root on one MI355X):", "", "```",
             "python3 bench.py --mode decode_split", "```", "",
             f"Each shape: {reps} calls captured in a graph per form, the two graphs replayed alternately "
             f"{rounds} times (median per call), weights rotated over >= {ROTATE_BYTES >> 20} MB of copies, "
             "random codes and scales. Round robin: the entry without a workspace (apex4_w4a4_gemm_tiled for "
             "G = 128 on tiled weights, apex4_w4a4_gemm for G = 32). Workspace: the same entry with the workspace "
             "the size query returns; it runs the stream-K form where the plan says decode_split, otherwise the "
             "same kernel as round robin (ratio ~1 there is the run-to-run spread).", "",
             "| G | K | N | M | plan (workspace entry) | workspace bytes | round robin µs | workspace µs | ratio |",
             "|---|---|---|---|---|---|---|---|---|"]
    for r_ in rows:
        lines.append(f"| {r_['G']} | {r_['K']} | {r_['N']} | {r_['M']} | {r_['plan_ws']} | {r_['workspace_bytes']} | "
                     f"{r_['round_robin_us']} | {r_['workspace_us']} | {r_['ratio']} |")
    with open(os.path.join(ROOT, "profiles", "decode_stream_k.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


def layers_mode(reps: int = 10):
    """The linears of one Llama-2-70B decoder layer under the uniform G=128 and the
    mixed configuration, each linear timed as quantize + W4A4 GEMM from fp16
    activations (apex4_w4a4_linear_ws), next to fp16 GEMMs of the same shapes
    (torch.matmul -> hipBLASLt).  Weights are rotated over at least 512 MB of
    copies (twice the Infinity Cache); codes and scales are random (speed does
    not depend on values).  The W4A4 linears are timed from a replayed graph of
    `reps` calls (GPU time, no Python launch overhead), the fp16 GEMMs eagerly.
    Each linear runs as W4A4Linear runs it: weights in the tiled layout for
    G >= 128 (row-major below), one apex4_w4a4_linear_ws call (the quantizer,
    then the GEMM, split over K or stream-K with a workspace where that
    applies)."""
    import torch
    import paper_2606_08761_amd as pk
    from paper_2606_08761_amd import workloads as wl
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)
    r = wl.rng_for("llama70b", 99)

    def timed(fn, n):
        for i in range(2):
            fn(i)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for i in range(n):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n * 1e3

    def graph_timed(fn, n):
        fn(0)
        torch.cuda.synchronize()
        side = torch.cuda.Stream(dev)
        side.wait_stream(stream)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            for i in range(n):
                fn(i)
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        del g
        return e0.elapsed_time(e1) / n * 1e3

    def copies(nbytes):
        return max(2, -(-ROTATE_BYTES // nbytes))

    for cfg, linears in LAYER_CONFIGS.items():
        wsets = {}
        for name, Nl, Kl, Gl in linears:
            Gv = Gl or Kl
            Wq = torch.from_numpy(wl.random_codes(r, Nl, Kl)).to(dev)
            if Gv >= 128:
                Wq = pk.apex4_tile_weights(Wq)
            sw = torch.from_numpy(wl.random_scales(r, Nl, Kl // Gv)).to(dev)
            R = copies(Nl * Kl // 2 + 2 * Nl * (Kl // Gv))
            wsets[name] = [(Wq, sw)] + [(Wq.clone(), sw.clone()) for _ in range(R - 1)]
        for Ml in LAYER_M:
            per, gbs, split = {}, {}, {}
            for name, Nl, Kl, Gl in linears:
                Gv = Gl or Kl
                x = torch.from_numpy(wl.activations(wl.rng_for("llama70b", 98, Ml + Kl), Ml, Kl)).to(dev)
                Y = torch.empty((Ml, Nl), dtype=torch.float16, device=dev)
                Aq = torch.empty((Ml, Kl // 2), dtype=torch.uint8, device=dev)
                sa = torch.empty((Ml, Kl // Gv), dtype=torch.float16, device=dev)
                ws = wsets[name]
                need = pk.apex4_w4a4_gemm_workspace_size(Ml, Nl, Kl, Gv)
                tiled = Gv >= 128
                # as W4A4Linear: one apex4_w4a4_linear_ws call (the quantizer, then
                # the GEMM, split over K or stream-K where a workspace applies)
                work = torch.empty((need,), dtype=torch.uint8, device=dev) if need else None

                def call(i):
                    pk.apex4_w4a4_linear_ws(x, ws[i % len(ws)][0], ws[i % len(ws)][1], Gv, workspace=work,
                                            tiled=tiled, Y=Y, A_q_work=Aq, s_a_work=sa, make_workspace=False)
                t = graph_timed(call, reps)
                # the workspace's use: S K ranges on the tile kernels, or the
                # stream-K form of the few-row kernel (reported as 0)
                kern_ws, s_ws = pk.apex4_w4a4_gemm_plan("gemm_ws", Ml, Nl, Kl, Gv,
                                                        pk.APEX4_DEBUG_W_TILED if tiled else 0)
                split[name] = 0 if kern_ws == "decode_split" else (s_ws if need else 1)
                per[name] = round(t, 2)
                # algorithmic HBM bytes of the linear: x, codes, scales, Y
                nbytes = 2 * Ml * Kl + Ml * Kl / 2 + Nl * Kl / 2 + 2 * (Ml + Nl) * Kl / Gv + 2 * Ml * Nl
                gbs[name] = round(nbytes / (t * 1e-6) / 1e9)
                del x, Y, Aq, sa
            print(json.dumps({"mode": "layers", "config": cfg, "M": Ml, "linear_us": per, "hbm_gbs": gbs,
                              "k_splits": split, "total_us": round(sum(per.values()), 2)}), flush=True)
        del wsets
        torch.cuda.empty_cache()
    # the MX variant: quantize_mx, then the MX GEMM (split over K with a workspace where it applies)
    for cfg, linears in MX_LAYER_CONFIGS.items():
        wsets = {}
        for name, Nl, Kl, Gl in linears:
            W6 = pk.apex4_pack_fp6(torch.from_numpy(wl.random_codes(r, Nl, Kl)).to(dev))
            ew = torch.from_numpy((127 + r.integers(-4, 2, size=(Nl, Kl // Gl))).astype(np.uint8)).to(dev)
            R = copies(3 * Nl * Kl // 4 + Nl * (Kl // Gl))
            wsets[name] = [(W6, ew)] + [(W6.clone(), ew.clone()) for _ in range(R - 1)]
        for Ml in LAYER_M:
            per, gbs, split = {}, {}, {}
            for name, Nl, Kl, Gl in linears:
                x = torch.from_numpy(wl.activations(wl.rng_for("llama70b", 98, Ml + Kl), Ml, Kl)).to(dev)
                Y = torch.empty((Ml, Nl), dtype=torch.float16, device=dev)
                A6 = torch.empty((Ml, 3 * Kl // 4), dtype=torch.uint8, device=dev)
                ea = torch.empty((Ml, Kl // Gl), dtype=torch.uint8, device=dev)
                ws = wsets[name]
                need = pk.apex4_w4a4_gemm_mx_workspace_size(Ml, Nl, Kl, Gl)
                work = torch.empty((max(need, 16),), dtype=torch.uint8, device=dev)

                def call(i):
                    pk.apex4_quantize_mx(x, Gl, A6, ea)
                    pk.apex4_w4a4_gemm_mx_ws(A6, ea, ws[i % len(ws)][0], ws[i % len(ws)][1], Gl, work, Y)
                t = graph_timed(call, reps)
                per[name] = round(t, 2)
                nbytes = 2 * Ml * Kl + 3 * Ml * Kl / 4 + 3 * Nl * Kl / 4 + (Ml + Nl) * Kl / Gl + 2 * Ml * Nl
                gbs[name] = round(nbytes / (t * 1e-6) / 1e9)
                split[name] = need // (4 * Ml * Nl) if need else 1
                del x, Y, A6, ea, work
            print(json.dumps({"mode": "layers", "config": cfg, "M": Ml, "linear_us": per, "hbm_gbs": gbs,
                              "k_splits": split, "total_us": round(sum(per.values()), 2)}), flush=True)
        del wsets
        torch.cuda.empty_cache()
    # fp16 GEMMs of the same shapes (the value projection is part of qkv)
    shapes = [("qkv", 10240, 8192), ("o", 8192, 8192), ("gate_up", 57344, 8192), ("down", 8192, 28672)]
    for Ml in LAYER_M:
        per = {}
        for name, Nl, Kl in shapes:
            wf = [torch.randn(Nl, Kl, dtype=torch.float16, device=dev) * 0.02 for _ in range(copies(2 * Nl * Kl))]
            x = torch.randn(Ml, Kl, dtype=torch.float16, device=dev)
            Y = torch.empty((Ml, Nl), dtype=torch.float16, device=dev)
            per[name] = round(timed(lambda i: torch.matmul(x, wf[i % len(wf)].t(), out=Y), reps), 2)
            del wf, x, Y
            torch.cuda.empty_cache()
        print(json.dumps({"mode": "layers", "config": "fp16", "M": Ml, "linear_us": per,
                          "total_us": round(sum(per.values()), 2)}), flush=True)


def summarize_layers(path, command):
    """profiles/layer_sweep_llama2_70b.md from the --mode layers output."""
    rows = [json.loads(l) for l in open(path) if l.startswith("{")]
    tot = {(r["config"], r["M"]): r for r in rows}
    lines = ["# Llama-2-70B decoder-layer linears: uniform G=128 vs mixed granularity vs fp16", "",
             "Command (run from the repository root on one MI355X):", "", "```", command, "```", "",
             "Each W4A4 linear is timed as W4A4Linear runs it: quantize + GEMM from fp16 activations in one "
             "apex4_w4a4_linear_ws call (tiled weights for G >= 128, row-major below; where the library asks "
             "for a workspace, the GEMM is split over K into S ranges on the tile kernels, marked S=, or runs "
             "the few-row kernel's stream-K form, marked stream-K) "
             "from a replayed graph (GPU time), weights rotated over >= 512 MB of copies; fp16 is "
             "torch.matmul (hipBLASLt) on the same shapes, rotated the same way, timed eagerly. "
             "mix: G=32 for the value and down projections, per-channel (G=K) elsewhere; q and k "
             "share one per-channel GEMM (N=9216).", "",
             "| M | g128 us | mix us | fp16 us | g128 speedup vs fp16 | mix speedup vs fp16 |",
             "|---|---|---|---|---|---|"]
    for Ml in sorted({r["M"] for r in rows}):
        g, mx, f = tot.get(("g128", Ml)), tot.get(("mix", Ml)), tot.get(("fp16", Ml))
        if not (g and mx and f):
            continue
        lines.append(f"| {Ml} | {g['total_us']} | {mx['total_us']} | {f['total_us']} | "
                     f"{f['total_us'] / g['total_us']:.2f} | {f['total_us'] / mx['total_us']:.2f} |")
    if any(r["config"].startswith("mx_") for r in rows):
        lines += ["", "MX variant (power-of-two group scales applied inside the FP6 MFMA, no per-group "
                  "dequantization; not the paper's fp16 scales): apex4_quantize_mx + apex4_w4a4_gemm_mx_ws.", "",
                  "| M | MX G=32 us | MX G=128 us | fp16 us | MX G=32 speedup vs fp16 | MX G=128 speedup vs fp16 |",
                  "|---|---|---|---|---|---|"]
        for Ml in sorted({r["M"] for r in rows}):
            a, b, f = tot.get(("mx_g32", Ml)), tot.get(("mx_g128", Ml)), tot.get(("fp16", Ml))
            if not (a and b and f):
                continue
            lines.append(f"| {Ml} | {a['total_us']} | {b['total_us']} | {f['total_us']} | "
                         f"{f['total_us'] / a['total_us']:.2f} | {f['total_us'] / b['total_us']:.2f} |")
    lines += ["", "Per linear (us; W4A4 rows also give the algorithmic HBM GB/s of x, codes, scales and Y):", "",
              "| config | M | per linear |", "|---|---|---|"]
    for r in rows:
        g, sp = r.get("hbm_gbs", {}), r.get("k_splits", {})
        lines.append(f"| {r['config']} | {r['M']} | " +
                     ", ".join(f"{k} {v}" + (f" ({g[k]} GB/s)" if k in g else "") +
                               (f" S={sp[k]}" if sp.get(k, 1) > 1 else "") +
                               (" stream-K" if sp.get(k, 1) == 0 else "") for k, v in r["linear_us"].items()) + " |")
    with open(os.path.join(ROOT, "profiles", "layer_sweep_llama2_70b.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


def _sq_means(paths, pick):
    """Mean per dispatch of every counter over the CSV rows whose kernel pick() accepts."""
    import csv
    import statistics
    vals = {}
    for p in paths:
        for r in csv.DictReader(open(p)):
            if pick(r["Kernel_Name"]):
                vals.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    return {k: statistics.mean(v) for k, v in vals.items()}


def _sq_section(c, what, mfma):
    """Where the SIMD cycles of one kernel go.  Quad-cycle counters are
    multiplied by 4; per-SIMD figures divide by the 1024 SIMDs; the kernel's
    cycle count is GRBM_GUI_ACTIVE over the 8 XCDs."""
    simds = 1024
    kcyc = c["GRBM_GUI_ACTIVE"] / 8
    quad = ["SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_ACTIVE_INST_ANY", "SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_VALU2",
            "SQ_ACTIVE_INST_LDS", "SQ_ACTIVE_INST_SCA", "SQ_ACTIVE_INST_MISC", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY",
            "SQ_WAIT_INST_LDS"]
    plain = ["SQ_VALU_MFMA_BUSY_CYCLES", "SQ_VALU_MFMA_COEXEC_CYCLES", "SQ_LDS_IDX_ACTIVE", "SQ_LDS_BANK_CONFLICT"]
    mf = c["SQ_INSTS_MFMA"] / simds
    lines = [f"Kernel length ({what}): GRBM_GUI_ACTIVE / 8 XCDs = {kcyc:.0f} cycles. Per SIMD: {mf:.0f} MFMA "
             f"({mfma}), {c['SQ_INSTS_VALU'] / simds:.0f} VALU "
             f"({c['SQ_INSTS_VALU'] / c['SQ_INSTS_MFMA']:.2f} per MFMA), {c['SQ_INSTS_LDS'] / simds:.0f} LDS, "
             f"{c.get('SQ_INSTS_SALU', 0) / simds:.0f} SALU instructions; {kcyc / mf:.1f} cycles per MFMA per SIMD.", "",
             "| counter | per SIMD (cycles) | share of kernel cycles |", "|---|---|---|"]
    for k in quad:
        if k in c:
            v = c[k] * 4 / simds
            lines.append(f"| {k} (quad-cycles x 4) | {v:.0f} | {v / kcyc:.3f} |")
    for k in plain:
        if k in c:
            v = c[k] / simds
            lines.append(f"| {k} | {v:.0f} | {v / kcyc:.3f} |")
    busy = (c["SQ_ACTIVE_INST_VALU"] * 4 + c["SQ_VALU_MFMA_BUSY_CYCLES"] - c["SQ_VALU_MFMA_COEXEC_CYCLES"]) / simds
    lines += ["", f"* cycles with a VALU or MFMA instruction executing (VALU + MFMA - co-executed): {busy:.0f} "
                  f"({busy / kcyc:.2f} of the kernel); VALU alone {c['SQ_ACTIVE_INST_VALU'] * 4 / simds / kcyc:.2f}, "
                  f"MFMA alone {c['SQ_VALU_MFMA_BUSY_CYCLES'] / simds / kcyc:.2f}",
              f"* VALU cycles per VALU instruction: {c['SQ_ACTIVE_INST_VALU'] * 4 / c['SQ_INSTS_VALU']:.2f}",
              "", "Raw means per dispatch:", "", "| counter | value |", "|---|---|"]
    lines += [f"| {k} | {c[k]:.4g} |" for k in sorted(c)]
    return lines


def summarize_sq(paths, cmds):
    """profiles/gemm_w4a4_sq_paper_shape.md: where the SIMD cycles of the
    paper-shape G=128 GEMM go, from SQ counters (means over the GEMM dispatches
    of bench.py --mode counters)."""
    c = _sq_means(paths, is_tiled_gemm)
    lines = [f"# W4A4 GEMM, M={M} N=K={N} G={G}: SQ counters (where the SIMD cycles go)", "",
             "Commands (run from the repository root on one MI355X):", "", "```", cmds, "```", ""]
    lines += _sq_section(c, "the G=128 GEMM", "v_mfma_i32_32x32x32_i8, 32 cycles at the MFMA peak")
    with open(os.path.join(ROOT, "profiles", "gemm_w4a4_sq_paper_shape.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


def summarize_sq_variants(paths, cmds):
    """profiles/gemm_variants_sq_paper_shape.md: the same SQ breakdown for the
    FP6-container and MX GEMMs (bench.py --mode variants)."""
    lines = [f"# FP6 and MX variant GEMMs, M={M} N=K={N} G={G}: SQ counters", "",
             "Commands (run from the repository root on one MI355X):", "", "```", cmds, "```", ""]
    for title, key, mfma in (("FP6 containers, fp16 scales (w4a4_gemm_fp6_kernel)", "gemm_fp6_kernel",
                              "v_mfma_scale_f32_32x32x64_f8f6f4, FP6 operands, unit scales"),
                             ("MX, power-of-two scales (w4a4_gemm_mx_kernel<4, 2>)", "gemm_mx_kernel",
                              "v_mfma_scale_f32_32x32x64_f8f6f4, FP6 operands, per-lane E8M0 scales")):
        c = _sq_means(paths, lambda n, key=key: key in n)
        if "GRBM_GUI_ACTIVE" in c and "SQ_INSTS_MFMA" in c:
            lines += [f"## {title}", ""] + _sq_section(c, title.split(" (")[0], mfma) + [""]
    with open(os.path.join(ROOT, "profiles", "gemm_variants_sq_paper_shape.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


# (label, M, N, K, G, tiled, kernel instantiation the plan picks: MROWS, ring depth, groups per stage)
DECODE_SQ = [("G=32, K=28672: the mixed configuration's down projection", 16, 8192, 28672, 32, False, "<16, 4, 4,"),
             ("G=128, N=K=8192, tiled weights", 16, 8192, 8192, 128, True, "<16, 6, 1,"),
             ("G=128, N=28672, K=8192, tiled weights, activations staged in LDS", 32, 28672, 8192, 128, True,
              "<32, 6, 1,")]


def decode_sq_mode(reps: int = 5):
    """Each DECODE_SQ few-row GEMM `reps` times (random codes and scales), for
    SQ counter passes; every case runs its own instantiation of the few-row
    kernel, which the summary tells apart by name."""
    import torch
    import paper_2606_08761_amd as pk
    from paper_2606_08761_amd import workloads as wl
    dev = torch.device("cuda", 0)
    for (label, Md, Nd, Kd, Gd, tiled, _) in DECODE_SQ:
        r = wl.rng_for("decode", 11, Md * 7 + Nd + Kd + Gd)
        Wq = torch.from_numpy(wl.random_codes(r, Nd, Kd)).to(dev)
        W = pk.apex4_tile_weights(Wq) if tiled else Wq
        sw = torch.from_numpy(wl.random_scales(r, Nd, Kd // Gd)).to(dev)
        Aq = torch.from_numpy(wl.random_codes(r, Md, Kd)).to(dev)
        sa = torch.from_numpy(wl.random_scales(r, Md, Kd // Gd)).to(dev)
        Y = torch.empty((Md, Nd), dtype=torch.float16, device=dev)
        for _ in range(reps):
            if tiled:
                pk.apex4_w4a4_gemm_tiled(Aq, sa, W, sw, Gd, None, Y)
            else:
                pk.apex4_w4a4_gemm(Aq, sa, W, sw, Gd, Y)
        torch.cuda.synchronize()
        plan = pk.apex4_w4a4_gemm_plan("gemm", Md, Nd, Kd, Gd, pk.APEX4_DEBUG_W_TILED if tiled else 0)
        print(json.dumps({"mode": "decode_sq", "case": label, "M": Md, "N": Nd, "K": Kd, "G": Gd, "plan": plan}),
              flush=True)


def summarize_decode_sq(paths, cmds):
    """profiles/decode_sq.md: where the SIMD cycles of the few-row kernel go
    (bench.py --mode decode_sq)."""
    lines = ["# Few-row GEMM (M = 16 and 32): SQ counters", "",
             "Commands (run from the repository root on one MI355X):", "", "```", cmds, "```", "",
             "Means over the launches of each case. The kernel fills the CUs with one 8-wave workgroup each; "
             "shares are of the kernel's cycles per SIMD.", ""]
    for (label, Md, Nd, Kd, Gd, tiled, key) in DECODE_SQ:
        c = _sq_means(paths, lambda n, key=key: "w4a4_decode_kernel" in n and key in n)
        if "GRBM_GUI_ACTIVE" in c and "SQ_INSTS_MFMA" in c:
            lines += [f"## M={Md} N={Nd} K={Kd} {label}", ""]
            lines += _sq_section(c, f"w4a4_decode_kernel{key.rstrip(',')}...>", "v_mfma_i32_32x32x32_i8") + [""]
    with open(os.path.join(ROOT, "profiles", "decode_sq.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


def summarize_power(path, command):
    """profiles/power_clock_paper_shape.md from the --mode power output."""
    rows = [json.loads(l) for l in open(path) if l.startswith("{")]
    lines = ["# Board power and shader clock under sustained GEMM load (M=2048, N=K=8192)", "",
             "Command (run from the repository root on one MI355X):", "", "```", command, "```", "",
             "Each kernel is launched back to back for about 3 s while amd-smi is sampled every 0.1 s "
             "(samples in the first 0.7 s are dropped). MI355X's board power limit is 1400 W; its peak "
             "shader clock is 2400 MHz.", "",
             "| kernel | us per launch | TOPS (2MNK/t) | socket power W (median) | mean gfx clock MHz (median) | samples |",
             "|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| {r['kernel']} | {r['us']} | {r['tops']} | {r['power_w']} | {r['clock_mhz']} | {r['samples']} |")
    with open(os.path.join(ROOT, "profiles", "power_clock_paper_shape.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


def power_mode(secs: float = 3.0):
    """Back-to-back launches of the paper-shape GEMMs for `secs` each while
    amd-smi samples socket power and the per-XCD gfx clocks."""
    import statistics
    import subprocess
    import threading
    import torch
    import paper_2606_08761_amd as pk
    from paper_2606_08761_amd import workloads as wl

    def sample():
        try:
            r = subprocess.run(["amd-smi", "metric", "-g", "0", "-p", "-c", "--json"], capture_output=True,
                               text=True, timeout=10)
            d = json.loads(r.stdout)
            g = d[0] if isinstance(d, list) else d["gpu_data"][0]
            pw = float(g["power"]["socket_power"]["value"])
            clks = [float(v["clk"]["value"]) for k, v in g["clock"].items()
                    if k.startswith("gfx_") and isinstance(v, dict) and isinstance(v.get("clk"), dict)]
            return pw, statistics.mean(clks) if clks else float("nan")
        except Exception:  # amd-smi missing or its format differs: no sample
            return None

    dev = torch.device("cuda", 0)
    cases = []
    for Gp in (G, K):
        c = [torch.from_numpy(a).to(dev) for a in wl.codes_workload("paper", M, N, K, Gp)]
        Y = torch.empty((M, N), dtype=torch.float16, device=dev)
        cases.append((f"W4A4 GEMM G={Gp}", (lambda c=c, Y=Y, Gp=Gp: pk.apex4_w4a4_gemm(*c, Gp, Y))))
    a8 = torch.randint(-128, 127, (M, K), dtype=torch.int8, device=dev)
    b8 = torch.randint(-128, 127, (K, N), dtype=torch.int8, device=dev)
    cases.append(("int8 GEMM, torch._int_mm (hipBLASLt), no scales", lambda: torch._int_mm(a8, b8)))
    x = torch.randn(M, K, dtype=torch.float16, device=dev)
    w = torch.randn(N, K, dtype=torch.float16, device=dev)
    cases.append(("fp16 GEMM, torch.matmul (hipBLASLt)", lambda: torch.matmul(x, w.t())))
    for name, fn in cases:
        fn()
        torch.cuda.synchronize()
        got, stop = [], [False]

        def loop():
            t0 = time.time()
            while not stop[0]:
                s_ = sample()
                if s_ is not None and time.time() - t0 > 0.7:
                    got.append(s_)
                time.sleep(0.1)

        th = threading.Thread(target=loop)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        th.start()
        n, t0 = 0, time.time()
        e0.record()
        while time.time() - t0 < secs:
            for _ in range(20):
                fn()
            n += 20
            torch.cuda.synchronize()
        e1.record()
        torch.cuda.synchronize()
        stop[0] = True
        th.join()
        us = e0.elapsed_time(e1) / n * 1e3
        pw = statistics.median([p for p, _ in got]) if got else None
        ck = statistics.median([c_ for _, c_ in got]) if got else None
        print(json.dumps({"mode": "power", "kernel": name, "us": round(us, 1), "tops": round(2.0 * M * N * K / us / 1e6),
                          "power_w": pw, "clock_mhz": None if ck is None else round(ck), "samples": len(got)}), flush=True)


def summarize_rho(path, command):
    """profiles/rho_probes.md from the rho probe output (shader-clock cycles, no profiler)."""
    r = json.load(open(path))
    co = r["mfma_cycles_per_simd_2_waves_v_fma_interleaved"]
    lines = ["# rho probes on MI355X (intra-CU INT8 MFMA vs fp32 VALU rates)", "",
             "Command (run from the repository root on one MI355X):", "", "```", command, "```", "",
             "Cycles are shader clocks counted inside the probe kernels (s_memtime); per-SIMD figures use the slowest "
             "wave of each CU.", "",
             "| quantity | value |", "|---|---|",
             f"| cycles per v_mfma_i32_32x32x32_i8 (1 wave/SIMD) | {r['cycles_per_mfma_i32_32x32x32_i8']:.2f} |",
             f"| INT8 MFMA ops/clk/CU | {r['int8_mfma_ops_per_clk_per_cu']:.0f} |",
             f"| cycles per v_fma_f32 per SIMD, 2 waves/SIMD | {r['cycles_per_v_fma_f32_per_simd_2_waves']:.2f} |",
             f"| cycles per v_fma_f32 per SIMD, 4 waves/SIMD | {r['cycles_per_v_fma_f32_per_simd_4_waves']:.2f} |",
             f"| fp32 flops/clk/CU (sustained) | {r['fp32_fma_flops_per_clk_per_cu_sustained']:.1f} |",
             f"| rho measured (INT8 MFMA ops / fp32 flops) | {r['rho_measured']:.1f} |",
             f"| rho datasheet, packed fp32 / unpacked | {r['rho_datasheet_packed_fp32']:.1f} / {r['rho_datasheet_unpacked_fp32']:.1f} |",
             f"| shader clock of the probe run (MHz) | {r['shader_clock_mhz']:.0f} |", "",
             "MFMA cycles per SIMD with 2 waves per SIMD, each interleaving V independent v_fma_f32 per MFMA:", "",
             "| V | " + " | ".join(co) + " |", "|---|" + "---|" * len(co),
             "| cycles | " + " | ".join(f"{v:.1f}" for v in co.values()) + " |"]
    with open(os.path.join(ROOT, "profiles", "rho_probes.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


def summarize_gsweep(trace_csv, pmc_csv, cmds):
    """profiles/gemm_w4a4_gsweep_m4096.md: per group size, kernel time and the
    VALU / MFMA instruction counts per wave and group (SQ counters).  GEMM
    dispatches are assigned to group sizes by position (GSWEEP_LAUNCHES each, in
    GSWEEP order)."""
    import csv
    import statistics
    Mg, Ng, Kg, Gs = GSWEEP
    waves = -(-Mg // 128) * -(-Ng // 256) * 8

    def by_position(ids):
        ids = sorted(ids)
        assert len(ids) == GSWEEP_LAUNCHES * len(Gs), (len(ids), "GEMM dispatches")
        return {d: Gs[i // GSWEEP_LAUNCHES] for i, d in enumerate(ids)}

    trace = [r for r in csv.DictReader(open(trace_csv)) if is_tiled_gemm(r["Kernel_Name"])]
    gmap = by_position({int(r["Dispatch_Id"]) for r in trace})
    durs = {}
    for r in trace:
        durs.setdefault(gmap[int(r["Dispatch_Id"])], []).append(
            (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    times = {g: statistics.median(v) for g, v in durs.items()}
    rows = [r for r in csv.DictReader(open(pmc_csv)) if is_tiled_gemm(r["Kernel_Name"])]
    pmap = by_position({int(r["Dispatch_Id"]) for r in rows})
    cnt = {}
    for r in rows:
        cnt.setdefault(pmap[int(r["Dispatch_Id"])], {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    c = {g: {k: statistics.mean(v) for k, v in d.items()} for g, d in cnt.items()}
    base_valu = c[Kg]["SQ_INSTS_VALU"]
    lines = [f"# W4A4 GEMM granularity sweep, M={Mg} N=K={Ng}: rocprofv3 summary", "",
             "Commands (run from the repository root on one MI355X):", "", "```", cmds, "```", "",
             "Per group and wave (one wave owns 128 x 32 outputs): MFMA cycles = MFMAs x 32 (v_mfma_i32_32x32x32_i8); "
             "dequant VALU cycles = (VALU instructions - those at G=K) x 4 (one wave64 VALU instruction per 4 SIMD cycles, "
             "measured). TOPS = 2MNK / median kernel time (kernel trace). For G < 128 a wave's group covers "
             "128/G times fewer MFMAs, so per-group counts are per the wave's 128 x 32 tile either way.", "",
             "| G | kernel us | TOPS | % INT8 peak | VALU/MFMA (instructions) | MFMA/wave/group | dequant VALU/wave/group "
             "| MFMA cycles/group | dequant VALU cycles/group | VALU/MFMA cycles |",
             "|---|---|---|---|---|---|---|---|---|---|"]
    for g in sorted(c):
        groups = Kg // g
        mf = c[g]["SQ_INSTS_MFMA"] / waves / groups
        dq = (c[g]["SQ_INSTS_VALU"] - base_valu) / waves / groups if g != Kg else 0.0
        t = times.get(g)
        tops = 2.0 * Mg * Ng * Kg / t / 1e6 if t else float("nan")
        lines.append(f"| {g} | {t:.1f} | {tops:.0f} | {100 * tops / INT8_PEAK_TOPS:.1f} | "
                     f"{c[g]['SQ_INSTS_VALU'] / c[g]['SQ_INSTS_MFMA']:.2f} | {mf:.0f} | {dq:.1f} | {mf * 32:.0f} | "
                     f"{dq * 4:.0f} | {dq * 4 / (mf * 32):.2f} |")
    lines += ["", "Raw SQ counters per dispatch (means):", "",
              "| G | " + " | ".join(sorted(next(iter(c.values())))) + " |",
              "|---|" + "---|" * len(next(iter(c.values())))]
    for g in sorted(c):
        lines.append(f"| {g} | " + " | ".join(f"{c[g][k]:.4g}" for k in sorted(c[g])) + " |")
    with open(os.path.join(ROOT, "profiles", "gemm_w4a4_gsweep_m4096.md"), "w") as f:
        f.write("\n".join(lines) + "\n")


def counters_mode():
    """Launch the paper-shape GEMM (tiled weights, as the bench times it) 3 times
    and a 256 MiB reference copy 3 times, nothing else, so that per-dispatch
    counters of both can be compared."""
    import torch
    import paper_2606_08761_amd as pk
    from paper_2606_08761_amd import rho, workloads as wl
    dev = torch.device("cuda", 0)
    c = [torch.from_numpy(a).to(dev) for a in wl.codes_workload("paper", M, N, K, G)]
    Wt = pk.apex4_tile_weights(c[2])                 # the bench's weight layout
    Y = torch.empty((M, N), dtype=torch.float16, device=dev)
    src = torch.randint(0, 255, (256 << 20,), dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        rho.copy(src, dst)
    for _ in range(3):
        pk.apex4_w4a4_gemm_tiled(c[0], c[1], Wt, c[3], G, Y=Y)
    torch.cuda.synchronize()
    print(json.dumps({"mode": "counters", "copy_bytes": 256 << 20, "gemm": [M, N, K, G],
                      "gemm_algorithmic_bytes": M * K // 2 + N * K // 2 + 2 * (M + N) * (K // G) + 2 * M * N}))


def variants_mode():
    """Launch the FP6-container and the MX GEMM (M=2048, N=K=8192, G=128) 3 times
    each, nothing else, for per-dispatch counters."""
    import torch
    import paper_2606_08761_amd as pk
    from paper_2606_08761_amd import workloads as wl
    dev = torch.device("cuda", 0)
    Aq, sa, Wq, sw = [torch.from_numpy(a).to(dev) for a in wl.codes_workload("paper", M, N, K, G)]
    A6, W6 = pk.apex4_pack_fp6(Aq), pk.apex4_pack_fp6(Wq)
    ea = torch.full((M, K // G), 127, dtype=torch.uint8, device=dev)
    ew = torch.full((N, K // G), 127, dtype=torch.uint8, device=dev)
    Y = torch.empty((M, N), dtype=torch.float16, device=dev)
    torch.cuda.synchronize()
    for _ in range(3):
        pk.apex4_w4a4_gemm_fp6(A6, sa, W6, sw, G, Y)
    for _ in range(3):
        pk.apex4_w4a4_gemm_mx(A6, ea, W6, ew, G, Y)
    torch.cuda.synchronize()
    print(json.dumps({"mode": "variants", "gemm": [M, N, K, G]}))


GSWEEP = (4096, 8192, 8192, (32, 64, 128, 256, 512, 1024, 8192))
GSWEEP_LAUNCHES = 23   # per group size: 3 warm-up + 20 timed


def gsweep_mode(reps: int = 20):
    """Granularity sweep (the paper's rho-aware group-size choice, Sec. 3.2.2):
    M=4096, N=K=8192, G in {32, 64, 128, 256, 512, 1024, K}, random codes and
    scales.  Exactly GSWEEP_LAUNCHES GEMM launches per G, in this order, so
    per-dispatch profiler records map to G by position."""
    import torch
    import paper_2606_08761_amd as pk
    from paper_2606_08761_amd import workloads as wl
    dev = torch.device("cuda", 0)
    Mg, Ng, Kg, Gs = GSWEEP
    stream = torch.cuda.current_stream(dev)
    for Gg in Gs:
        c = [torch.from_numpy(a).to(dev) for a in wl.codes_workload("gsweep", Mg, Ng, Kg, Gg)]
        Y = torch.empty((Mg, Ng), dtype=torch.float16, device=dev)
        for _ in range(GSWEEP_LAUNCHES - reps):
            pk.apex4_w4a4_gemm(*c, Gg, Y)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            pk.apex4_w4a4_gemm(*c, Gg, Y)
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / reps * 1e3
        print(json.dumps({"mode": "gsweep", "M": Mg, "N": Ng, "K": Kg, "G": Gg, "us": round(us, 2),
                          "tops": round(2.0 * Mg * Ng * Kg / us / 1e6, 1), "launches": GSWEEP_LAUNCHES}), flush=True)
        del c, Y


# (M, N, K): Llama-2-70B o_proj-sized (8192 x 8192), gate/up-sized (28672 x
# 8192) and down (8192 x 28672) linears at decode batch sizes
DECODE_CASES = ([(M_, N_, 8192) for N_ in (8192, 28672) for M_ in (1, 8, 32)] + [(1, 8192, 28672), (8, 8192, 28672)] +
                [(16, 10240, 8192), (16, 8192, 8192), (16, 57344, 8192), (16, 8192, 28672)])  # Llama-2-70B at M = 16


def decode_bench(reps: int = 50):
    """Decode-size linears (few rows, memory-bound): quantize + GEMM from fp16 x,
    with the weights in the tiled layout (what W4A4Linear keeps); the same
    calls on row-major weights are reported beside them.

    Weight copies are rotated past the 256 MB Infinity Cache.  Algorithmic bytes of
    the GEMM: M K/2 + N K/2 + 2 (M + N) K/G + 2 M N; the linear adds the fp16 x
    (2 M K).  Also times the fp16 GEMM of the same shape (torch -> hipBLASLt).
    Each W4A4 call is timed twice: eager (one Python call per launch, which at
    these sizes is partly launch-bound) and as a replayed graph of the same
    calls (GPU time; the HBM rates use it).
    """
    import torch
    import paper_2606_08761_amd as pk
    from paper_2606_08761_amd import rho as rho_probe
    from paper_2606_08761_amd import workloads as wl
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)
    out = []
    wcache = {}
    for (Md, Nd, Kd) in DECODE_CASES:
        Gd = 128
        if (Nd, Kd) not in wcache:
            w = torch.from_numpy(wl.weights(wl.rng_for("decode", 2, Nd), Nd, Kd)).to(dev)
            Wq, sw = pk.apex4_quantize_act(w, Gd)
            Rw = max(2, -(-ROTATE_BYTES // (Nd * Kd // 2 + 2 * Nd * (Kd // Gd))))
            Rf = max(2, -(-ROTATE_BYTES // (2 * Nd * Kd)))
            wcache.clear()
            Wt = pk.apex4_tile_weights(Wq)
            wcache[(Nd, Kd)] = ([(Wq.clone(), sw.clone()) for _ in range(Rw)], [w.clone() for _ in range(Rf)],
                                [Wt.clone() for _ in range(Rw)])
            del w, Wq, sw, Wt
        qsets, fsets, tsets = wcache[(Nd, Kd)]
        x = torch.from_numpy(wl.activations(wl.rng_for("decode", 1, Md * 1000 + Nd // 1024), Md, Kd)).to(dev)
        Aq = torch.empty((Md, Kd // 2), dtype=torch.uint8, device=dev)
        sa = torch.empty((Md, Kd // Gd), dtype=torch.float16, device=dev)
        Y = torch.empty((Md, Nd), dtype=torch.float16, device=dev)
        pk.apex4_quantize_act(x, Gd, Aq, sa)

        def timed(fn):
            for i in range(5):
                fn(i)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            for i in range(reps):
                fn(i)
            e1.record(stream)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / reps * 1e3

        def graph_timed(fn, out):
            """GPU time per call without the Python launch overhead: `reps` calls
            captured in one graph, replayed; the replayed output must equal the
            eager output bit for bit (the kernels are deterministic)."""
            fn(reps - 1)
            torch.cuda.synchronize()
            ref = out.clone()
            side = torch.cuda.Stream(dev)
            side.wait_stream(stream)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                for i in range(reps):
                    fn(i)
            out.zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            if not torch.equal(out, ref):
                raise RuntimeError("graph replay differs from the eager result")
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            g.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            del g
            return e0.elapsed_time(e1) / reps * 1e3

        nq = len(qsets)
        lin = lambda i: pk.apex4_w4a4_linear_tiled(x, tsets[i % nq], qsets[i % nq][1], Gd, Y, Aq, sa)
        gem = lambda i: pk.apex4_w4a4_gemm_tiled(Aq, sa, tsets[i % nq], qsets[i % nq][1], Gd, Y=Y)
        lin_r = lambda i: pk.apex4_w4a4_linear(x, qsets[i % nq][0], qsets[i % nq][1], Gd, Y, Aq, sa)
        gem_r = lambda i: pk.apex4_w4a4_gemm(Aq, sa, qsets[i % nq][0], qsets[i % nq][1], Gd, Y)
        lin_us = timed(lin)
        gemm_us = timed(gem)
        lin_g_us = graph_timed(lin, Y)
        gemm_g_us = graph_timed(gem, Y)
        lin_r_g_us = graph_timed(lin_r, Y)
        gemm_r_g_us = graph_timed(gem_r, Y)
        # the same linear as two kernels (quantizer, then GEMM): what the linear
        # entry point runs unless its one-row fused kernel pays
        two = lambda i: (pk.apex4_quantize_act(x, Gd, Aq, sa), gem(i))
        two_g_us = graph_timed(two, Y)
        # a plain streaming read of the same weight copies: the speed any kernel
        # that reads these bytes once reaches at this size (the practical roofline)
        sink = torch.zeros(1024, dtype=torch.int32, device=dev)
        read_g_us = graph_timed(lambda i: rho_probe.read(tsets[i % nq], sink), sink)
        read_bytes = tsets[0].numel()
        yf = torch.empty((Md, Nd), dtype=torch.float16, device=dev)
        fp16_us = timed(lambda i: torch.matmul(x, fsets[i % len(fsets)].t(), out=yf))
        gbytes = Md * Kd / 2 + Nd * Kd / 2 + 2 * (Md + Nd) * Kd / Gd + 2 * Md * Nd
        out.append({"M": Md, "N": Nd, "K": Kd, "G": Gd, "linear_us": round(lin_us, 2), "gemm_us": round(gemm_us, 2),
                    "linear_graph_us": round(lin_g_us, 2), "gemm_graph_us": round(gemm_g_us, 2),
                    "quant_then_gemm_graph_us": round(two_g_us, 2),
                    "gemm_hbm_gbs": round(gbytes / (gemm_g_us * 1e-6) / 1e9, 1),
                    "gemm_hbm_frac": round(gbytes / (gemm_g_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 3),
                    "linear_hbm_gbs": round((gbytes + 2 * Md * Kd) / (lin_g_us * 1e-6) / 1e9, 1),
                    "kernel": pk.apex4_w4a4_gemm_plan("linear", Md, Nd, Kd, Gd, pk.APEX4_DEBUG_W_TILED)[0],
                    "row_major_linear_graph_us": round(lin_r_g_us, 2), "row_major_gemm_graph_us": round(gemm_r_g_us, 2),
                    "row_major_gemm_hbm_frac": round(gbytes / (gemm_r_g_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 3),
                    "read_graph_us": round(read_g_us, 2),
                    "read_hbm_frac": round(read_bytes / (read_g_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 3),
                    "gemm_rate_vs_read": round(read_g_us / gemm_g_us, 3),
                    "fp16_gemm_us": round(fp16_us, 2), "speedup_linear_vs_fp16": round(fp16_us / lin_us, 3),
                    "speedup_linear_graph_vs_fp16": round(fp16_us / lin_g_us, 3)})
        del x, Aq, sa, Y, yf
    wcache.clear()
    torch.cuda.synchronize()
    return out


# Decode-size linears for per-kernel HBM traffic counters: the memory-bound
# configuration (M in {1, 8, 32}, N x K = 8192 x 8192 and 28672 x 8192) and the
# Llama-2-70B linears at M = 16; G = 128.
DECODE_TRAFFIC = ([("decode", Md, Nd, 8192) for Nd in (8192, 28672) for Md in (1, 8, 32)] +
                  [("llama70b M=16 qkv", 16, 10240, 8192), ("llama70b M=16 o_proj", 16, 8192, 8192),
                   ("llama70b M=16 gate_up", 16, 57344, 8192), ("llama70b M=16 down", 16, 8192, 28672)])
DECODE_TRAFFIC_REPS = 3


def decode_counters_mode():
    """A 256 MiB reference copy 3 times, then each DECODE_TRAFFIC linear
    (apex4_w4a4_linear_tiled from fp16 x: the fused one-row kernel where it
    applies, else the quantizer and the GEMM) DECODE_TRAFFIC_REPS times, on
    tiled weight copies rotated past the 256 MB cache (after one pass over
    every copy).  All inputs are made and that pass is done first, so the
    kernels after the first copy are exactly these, in order; the printed
    launch list maps profiler dispatches to cases."""
    import torch
    import paper_2606_08761_amd as pk
    from paper_2606_08761_amd import rho, workloads as wl
    dev = torch.device("cuda", 0)
    Gd = 128
    src = torch.randint(0, 255, (256 << 20,), dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    cases = []
    for (label, Md, Nd, Kd) in DECODE_TRAFFIC:
        w = torch.from_numpy(wl.weights(wl.rng_for("decode", 2, Nd * 3 + Kd // 1024), Nd, Kd)).to(dev)
        Wq, sw = pk.apex4_quantize_act(w, Gd)
        # tiled copies rotated past the 256 MB cache (each launch reads weights
        # no recent launch touched)
        R = max(2, -(-ROTATE_BYTES // (Nd * Kd // 2)))
        Wts = [pk.apex4_tile_weights(Wq) for _ in range(R)]
        del w, Wq
        x = torch.from_numpy(wl.activations(wl.rng_for("decode", 1, Md * 1000 + Nd // 1024), Md, Kd)).to(dev)
        bufs = (torch.empty((Md, Nd), dtype=torch.float16, device=dev),
                torch.empty((Md, Kd // 2), dtype=torch.uint8, device=dev),
                torch.empty((Md, Kd // Gd), dtype=torch.float16, device=dev))
        kern, _ = pk.apex4_w4a4_gemm_plan("linear", Md, Nd, Kd, Gd, pk.APEX4_DEBUG_W_TILED)
        cases.append((label, Md, Nd, Kd, kern, x, Wts, sw, bufs))
    # one untraced pass over every copy (address translation warm), in the
    # rotation order, so each traced launch reads weights evicted from the cache
    for (label, Md, Nd, Kd, kern, x, Wts, sw, (Y, Aq, sa)) in cases:
        for Wt in Wts:
            pk.apex4_w4a4_linear_tiled(x, Wt, sw, Gd, Y, Aq, sa)
    torch.cuda.synchronize()
    launches = []
    for _ in range(3):
        rho.copy(src, dst)
        launches.append(("copy", "copy", 256 << 20, 256 << 20))
    for (label, Md, Nd, Kd, kern, x, Wts, sw, (Y, Aq, sa)) in cases:
        wbytes = Nd * Kd // 2 + 2 * Nd * (Kd // Gd)
        for i in range(DECODE_TRAFFIC_REPS):
            pk.apex4_w4a4_linear_tiled(x, Wts[i % len(Wts)], sw, Gd, Y, Aq, sa)
            tag = label if label != "decode" else f"decode M={Md} N={Nd} K={Kd}"
            if kern == "fused":
                launches.append((tag, "fused", 2 * Md * Kd + wbytes, 2 * Md * Nd + Md * Kd // 2 + 2 * Md * (Kd // Gd)))
            else:
                launches.append((tag, "quant", 2 * Md * Kd, Md * Kd // 2 + 2 * Md * (Kd // Gd)))
                launches.append((tag, kern, Md * Kd // 2 + 2 * Md * (Kd // Gd) + wbytes, 2 * Md * Nd))
    torch.cuda.synchronize()
    print(json.dumps({"mode": "decode_counters", "G": Gd, "launches": launches}), flush=True)


def _decode_kernel_role(name: str):
    """Role of a profiled dispatch in --mode decode_counters, or None for others."""
    if "copy_kernel" in name:
        return "copy"
    if "quant_small_kernel" in name or "quant_large_kernel" in name:
        return "quant"
    m = re.search(r"w4a4_gemv(?:_tiled)?_kernel<(true|false)", name)
    if m:
        return "fused" if m.group(1) == "true" else "gemv"
    if "w4a4_decode_kernel" in name:
        return "decode"
    if is_tiled_gemm(name):
        return "tile"
    return None


def summarize_decode_traffic(args):
    """profiles/decode_traffic.md: HBM bytes per dispatch of the decode-size
    linears (FETCH_SIZE and WRITE_SIZE, scaled by what they read for the
    256 MiB reference copy) next to the algorithmic bytes and the kernel-trace
    durations of the same launches."""
    import csv
    import statistics
    log = json.loads([l for l in open(args.decode_log) if l.startswith("{")][-1])
    launches = log["launches"]

    def ordered(path, counter=None, name_key="Kernel_Name"):
        rows = []
        for r in csv.DictReader(open(path)):
            if counter and r.get("Counter_Name") != counter:
                continue
            role = _decode_kernel_role(r[name_key])
            if role is None:
                continue
            rows.append((int(r.get("Dispatch_Id") or r.get("Correlation_Id") or 0), role, r))
        rows.sort(key=lambda t: t[0])
        # set-up (weight quantization) precedes the first reference copy
        first = next(i for i, t in enumerate(rows) if t[1] == "copy")
        rows = rows[first:]
        if [t[1] for t in rows] != [l[1] for l in launches]:
            raise SystemExit(f"{path}: dispatch roles {[t[1] for t in rows]} differ from the launch list")
        return [t[2] for t in rows]

    fetch = [float(r["Counter_Value"]) for r in ordered(args.decode_fetch_csv, "FETCH_SIZE")]
    write = [float(r["Counter_Value"]) for r in ordered(args.decode_write_csv, "WRITE_SIZE")]
    trace = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in ordered(args.decode_trace_csv)]
    kib = (256 << 20) / 1024.0
    fs = kib / statistics.mean(fetch[:3])
    ws = kib / statistics.mean(write[:3])
    groups = {}
    for (tag, role, rb, wb), f, w, us in zip(launches, fetch, write, trace):
        if role == "copy":
            continue
        g = groups.setdefault((tag, role), dict(rb=rb, wb=wb, f=[], w=[], us=[]))
        g["f"].append(f * fs * 1024.0)
        g["w"].append(w * ws * 1024.0)
        g["us"].append(us)
    cmds = open(args.decode_commands).read().strip() if args.decode_commands else ""
    lines = ["# Decode-size linears: HBM traffic per kernel (rocprofv3 counters)", "",
             "Commands (run from the repository root on one MI355X):", "", "```", cmds, "```", "",
             "`bench.py --mode decode_counters` runs a 256 MiB reference copy 3 times, then each linear",
             "(`apex4_w4a4_linear_tiled` from fp16 x, G = 128: the fused one-row kernel where the library picks",
             "it, else the quantizer and the GEMM) 3 times, on tiled weight copies rotated past the 256 MB cache",
             "(every copy is used once, untraced, before the reference copy).",
             "FETCH_SIZE and WRITE_SIZE",
             "(KiB per dispatch) are scaled by what they read for the copy "
             f"(read scale {fs:.3f}, write scale {ws:.3f}).  Duration: kernel trace of a separate run of the same",
             "command (mean of the 3 launches; counter runs serialize dispatches).  GB/s = (measured read + write)",
             "/ duration; algorithmic bytes: codes, scales, fp16 x or Y as the kernel must move them once.", "",
             "| linear | kernel | algorithmic read MB | HBM read MB | algorithmic write MB | HBM write MB | "
             "measured / algorithmic | duration us | HBM GB/s | fraction of 8 TB/s |",
             "|---|---|---|---|---|---|---|---|---|---|"]
    for (tag, role), g in groups.items():
        rd, wr, us = statistics.mean(g["f"]), statistics.mean(g["w"]), statistics.mean(g["us"])
        gbs = (rd + wr) / (us * 1e-6) / 1e9
        lines.append(f"| {tag} | {role} | {g['rb'] / 1e6:.2f} | {rd / 1e6:.2f} | {g['wb'] / 1e6:.3f} | {wr / 1e6:.3f} | "
                     f"{(rd + wr) / (g['rb'] + g['wb']):.2f} | {us:.2f} | {gbs:.0f} | {gbs / HBM_PEAK_GBS:.3f} |")
    with open(os.path.join(ROOT, "profiles", "decode_traffic.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    args = parse()
    if args.mode == "counters":
        return counters_mode()
    if args.mode == "summarize":
        return summarize_mode(args)
    if args.mode == "gsweep":
        return gsweep_mode()
    if args.mode == "power":
        return power_mode()
    if args.mode == "layers":
        return layers_mode()
    if args.mode == "variants":
        return variants_mode()
    if args.mode == "decode_counters":
        return decode_counters_mode()
    if args.mode == "decode_split":
        return decode_split_mode()
    if args.mode == "decode_sq":
        return decode_sq_mode()
    if args.mode == "rho":
        from paper_2606_08761_amd import rho
        print(json.dumps(rho.measure()), flush=True)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this benchmark runs on exactly one GPU; --gpus must be 1 "
              "(the path shards over rows, or over N and K on group boundaries, but no multi-GPU code is built)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2606_08761_amd as pk
    from paper_2606_08761_amd import workloads as wl

    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)

    # ---- inputs: fp16 activations and offline-quantized weights, R rotating copies ----
    x_h, w_h = wl.float_workload("paper", M, N, K)
    per_set = M * K * 2 + N * K // 2 + N * (K // G) * 2 + M * N * 2 + M * K // 2 + M * (K // G) * 2
    R = max(2, -(-ROTATE_BYTES // per_set))
    sets = []
    w_dev = torch.from_numpy(w_h).to(dev)
    Wq0, sw0 = pk.apex4_quantize_act(w_dev, G)
    Wt0 = pk.apex4_tile_weights(Wq0)                     # offline weight packing (tiled layout)
    for r in range(R):
        x = torch.from_numpy(x_h).to(dev)
        if r:
            x = x.roll(r, dims=0).contiguous()           # different bytes per set, same distribution
        sets.append(dict(x=x, Wq=Wq0.clone(), Wt=Wt0.clone(), sw=sw0.clone(),
                         Y=torch.empty((M, N), dtype=torch.float16, device=dev),
                         Aq=torch.empty((M, K // 2), dtype=torch.uint8, device=dev),
                         sa=torch.empty((M, K // G), dtype=torch.float16, device=dev)))
    del w_dev
    torch.cuda.synchronize()

    def step(i, marks=None):
        s = sets[i % R]
        if marks is not None:
            marks[2 * i].record(stream)
        pk.apex4_quantize_act(s["x"], G, s["Aq"], s["sa"])
        if marks is not None:
            marks[2 * i + 1].record(stream)
        pk.apex4_w4a4_gemm_tiled(s["Aq"], s["sa"], s["Wt"], s["sw"], G, Y=s["Y"])

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # ---- timed region: exactly `steps` steps ----
    # Two timing marks per step on the stream both kernels run on: before the
    # quantizer and between it and the GEMM; the GEMM of step i ends at the
    # first mark of step i + 1 (the stream runs in order), the last at a final
    # mark.
    try:
        marks = [TimingEvent() for _ in range(2 * args.steps + 1)]
        timing_marks = "hipEventDisableSystemFence events, 2 per step"
    except (OSError, AttributeError, RuntimeError) as e:  # the runtime refused the flag: torch's events
        print(f"bench.py: fence-free timing events unavailable ({e}); using torch.cuda.Event", file=sys.stderr)
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(2 * args.steps + 1)]
        timing_marks = "torch.cuda.Event (system-scope fence at each record), 2 per step"
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i, marks)
    marks[2 * args.steps].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    quant_ms = float(np.mean([marks[2 * i].elapsed_time(marks[2 * i + 1]) for i in range(args.steps)]))
    gemm_all = [marks[2 * i + 1].elapsed_time(marks[2 * i + 2]) for i in range(args.steps)]
    for e in marks:
        if isinstance(e, TimingEvent):
            e.destroy()
    gemm_ms = float(np.mean(gemm_all))
    ms_per_step = wall * 1e3 / args.steps
    ops = 2.0 * M * N * K
    value = ops / (ms_per_step * 1e-3) / 1e12
    gemm_tops = ops / (gemm_ms * 1e-3) / 1e12

    # ---- GEMM alone on the random-code workload (value-independent speed check) ----
    Aq_h, sa_h, Wq_h, sw_h = wl.codes_workload("paper", M, N, K, G)
    c = [torch.from_numpy(a).to(dev) for a in (Aq_h, sa_h, Wq_h, sw_h)]
    Wt_c = pk.apex4_tile_weights(c[2])
    Yc = torch.empty((M, N), dtype=torch.float16, device=dev)
    Yt = torch.empty_like(Yc)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 20

    def avg_ms(fn):
        for _ in range(5):
            fn()
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    codes_gemm_ms = avg_ms(lambda: pk.apex4_w4a4_gemm(*c, G, Yc))           # row-major weights
    codes_gemm_t_ms = avg_ms(lambda: pk.apex4_w4a4_gemm_tiled(c[0], c[1], Wt_c, c[3], G, Y=Yt))
    rowmajor_step_gemm_ms = avg_ms(lambda: pk.apex4_w4a4_gemm(sets[0]["Aq"], sets[0]["sa"], sets[0]["Wq"],
                                                              sets[0]["sw"], G, sets[0]["Y"]))
    tiled_same_bits = bool(torch.equal(Yc, Yt))
    del Wt_c, Yt

    # ---- the same GEMM on the FP6 matrix cores (codes re-encoded as e3m2) ----
    A6, W6 = pk.apex4_pack_fp6(c[0]), pk.apex4_pack_fp6(c[2])
    Y6 = torch.empty_like(Yc)
    for _ in range(5):
        pk.apex4_w4a4_gemm_fp6(A6, c[1], W6, c[3], G, Y6)
    e0.record(stream)
    for _ in range(reps):
        pk.apex4_w4a4_gemm_fp6(A6, c[1], W6, c[3], G, Y6)
    e1.record(stream)
    torch.cuda.synchronize()
    fp6_ms = e0.elapsed_time(e1) / reps
    e0.record(stream)
    for _ in range(reps):
        pk.apex4_pack_fp6(c[0], A6)
    e1.record(stream)
    torch.cuda.synchronize()
    pack_ms = e0.elapsed_time(e1) / reps
    fp6 = {"gemm_us": round(fp6_ms * 1e3, 3), "tops": round(2.0 * M * N * K / (fp6_ms * 1e-3) / 1e12, 2),
           "time_vs_int8_kernel": round(fp6_ms / codes_gemm_ms, 3),
           "same_bits_as_int8_kernel": bool(torch.equal(Y6.view(torch.int16), Yc.view(torch.int16))),
           "pack_activations_us": round(pack_ms * 1e3, 3),
           "mfma": "v_mfma_scale_f32_32x32x64_f8f6f4, FP6 e3m2 operands, unit E8M0 scales"}
    del c, Yc, A6, W6, Y6

    # ---- MX variant: power-of-two group scales applied inside the FP6 MFMA ----
    # (a different quantization: its accuracy cost is reported next to the
    # fp16-scale path's, both against an fp32 GEMM of the unquantized inputs)
    xm, w16 = sets[0]["x"], torch.from_numpy(w_h).to(dev)
    A6m, eam = pk.apex4_quantize_mx(xm, G)
    W6m, ewm = pk.apex4_quantize_mx(w16, G)
    Ym = torch.empty((M, N), dtype=torch.float16, device=dev)
    for _ in range(5):
        pk.apex4_w4a4_gemm_mx(A6m, eam, W6m, ewm, G, Ym)
    e0.record(stream)
    for _ in range(reps):
        pk.apex4_w4a4_gemm_mx(A6m, eam, W6m, ewm, G, Ym)
    e1.record(stream)
    torch.cuda.synchronize()
    mx_ms = e0.elapsed_time(e1) / reps
    e0.record(stream)
    for _ in range(reps):
        pk.apex4_quantize_mx(xm, G, A6m, eam)
    e1.record(stream)
    torch.cuda.synchronize()
    mxq_ms = e0.elapsed_time(e1) / reps
    ref = xm.float() @ w16.float().t()
    rms = lambda t: float(t.double().pow(2).mean().sqrt())
    pk.apex4_quantize_act(xm, G, sets[0]["Aq"], sets[0]["sa"])
    pk.apex4_w4a4_gemm(sets[0]["Aq"], sets[0]["sa"], sets[0]["Wq"], sets[0]["sw"], G, sets[0]["Y"])
    mx = {"gemm_us": round(mx_ms * 1e3, 3), "tops": round(2.0 * M * N * K / (mx_ms * 1e-3) / 1e12, 2),
          "time_vs_fp16_scale_kernel": round(mx_ms / codes_gemm_ms, 3), "quantize_us": round(mxq_ms * 1e3, 3),
          "rel_rms_err_vs_fp32": round(rms(Ym.float() - ref) / rms(ref), 5),
          "fp16_scale_rel_rms_err_vs_fp32": round(rms(sets[0]["Y"].float() - ref) / rms(ref), 5),
          "scales": "E8M0 powers of two (smallest covering max|x|/7), not the paper's fp16 scales",
          "mfma": "v_mfma_scale_f32_32x32x64_f8f6f4, FP6 e3m2 codes, per-lane E8M0 group scales"}
    del A6m, W6m, Ym, ref, w16

    # ---- fp16 GEMM of the same shape (torch -> hipBLASLt), rotated too ----
    fsets = []
    Rf = max(2, -(-ROTATE_BYTES // (M * K * 2 + N * K * 2 + M * N * 2)))
    wf = torch.from_numpy(w_h).to(dev)
    for r in range(Rf):
        fsets.append((torch.from_numpy(x_h).to(dev), wf.clone(), torch.empty((M, N), dtype=torch.float16, device=dev)))
    for i in range(5):
        xf, wff, yf = fsets[i % Rf]
        torch.matmul(xf, wff.t(), out=yf)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(reps):
        xf, wff, yf = fsets[i % Rf]
        torch.matmul(xf, wff.t(), out=yf)
    e1.record(stream)
    torch.cuda.synchronize()
    fp16_ms = e0.elapsed_time(e1) / reps
    del fsets, wf

    line = {
        "metric": "W4A4-g128 GEMM TOPS + speedup vs fp16 GEMM, M=2048 N=K=8192; % INT8 MFMA peak",
        "value": round(value, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int4",
        "data": "synthetic",
        "config": {"workload": "W4A4-g128 linear, paper GEMM shape: quantize fp16 x[2048,8192] "
                               "(SymQuant, G=128) + W4A4 GEMM against W_q[8192,8192] (tiled weight layout)",
                   "M": M, "N": N, "K": K, "G": G, "parallelism": "none (1 GPU)",
                   "mfma": "v_mfma_i32_32x32x32_i8, i32 group sums, fp32 dequant, fp16 out",
                   "rotating_input_sets": R},
        "roofline": {"bound": "mfma", "achieved": round(gemm_tops, 2), "peak": INT8_PEAK_TOPS,
                     "unit": "TOP/s", "frac": round(gemm_tops / INT8_PEAK_TOPS, 4),
                     "traffic": traffic_from_profile(), "kernel": "w4a4_gemm_pp_kernel",
                     "kernel_us": round(gemm_ms * 1e3, 3)},
        "timing_marks": timing_marks,
        "quant_us": round(quant_ms * 1e3, 3),
        "quant_hbm_gbs": round((2.5 * M * K + 2 * M * K / G) / (quant_ms * 1e-3) / 1e9, 1),
        "gemm_us": round(gemm_ms * 1e3, 3),
        "gemm_us_p10_p50_p90": [round(float(np.percentile(gemm_all, q)) * 1e3, 3) for q in (10, 50, 90)],
        "gemm_tops": round(gemm_tops, 2),
        "gemm_pct_int8_peak": round(100 * gemm_tops / INT8_PEAK_TOPS, 2),
        "gemm_random_codes_us": round(codes_gemm_t_ms * 1e3, 3),
        "weights": "tiled layout (apex4_tile_weights, offline)",
        "gemm_row_major_weights_us": round(rowmajor_step_gemm_ms * 1e3, 3),
        "gemm_random_codes_row_major_us": round(codes_gemm_ms * 1e3, 3),
        "tiled_same_bits_as_row_major": tiled_same_bits,
        "fp16_gemm_us": round(fp16_ms * 1e3, 3),
        "fp16_gemm_tflops": round(ops / (fp16_ms * 1e-3) / 1e12, 2),
        "speedup_gemm_vs_fp16": round(fp16_ms / gemm_ms, 3),
        "speedup_step_vs_fp16": round(fp16_ms / ms_per_step, 3),
        "fp6_variant": fp6,
        "mx_variant": mx,
    }
    if not args.no_decode:
        line["decode"] = decode_bench()
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(args.cpu_seconds)
        # the same oracle on one host thread (a shorter sample)
        line["cpu_baseline_1thread"] = cpu_baseline(args.cpu_seconds / 2, threads=1)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
