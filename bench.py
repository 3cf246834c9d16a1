"""Benchmark of the lattice hot path on one MI355X.

One step = one pass of the whole path over one synthetic cloud: create the
lattice (embed, hash, vertex lists, neighbour table), splat, the lattice
convolutions of every level (1-hop, strided Downsample, transposed
Upsample), coarsening, slice and DeformSlice.  Inputs are resident in HBM
before timing starts.  Default workload: the 120,000-point LiDAR-like scan
(sigma 0.3 m, three lattice levels, fp32).

Prints one JSON line with the throughput (points/s), the roofline position
of the dominant kernel family (timed with HIP events on its launch stream
inside the timed region) and the CPU oracle's throughput on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"hbm": 8.0e12, "mfma_f32": 157.3e12, "mfma_bf16": 2.5e15}
FAMILIES = ["fill", "insert", "scan", "lists", "nbr", "splat", "conv", "slice", "deform_slice"]


def conv_flops(wl, levels):
    """Nominal flops of all convolutions of one step (9 taps each)."""
    total = 0
    for op in wl.ops:
        if op["op"] in ("conv", "conv_down", "refine"):
            n_out = levels[op["level"]].n
            total += 2 * n_out * 9 * op["src"][2] * op["dst"][2]
    return total


def algorithmic_bytes(wl, levels, family):
    """Bytes a kernel family must move per step (each input read once, each
    output written once), for the HBM-bound families."""
    u = 2 if wl.dtype == "bf16" else 4
    m = wl.m
    if family == "splat":
        C = next(op["dst"][2] for op in wl.ops if op["op"] == "splat")
        n = levels[0].n
        # features m*C*u, lists 4m*(4 entry + 4 weight), offsets, output n*C*u
        return m * C * u + 4 * m * 8 + (n + 1) * 4 + n * C * u
    if family in ("slice", "deform_slice"):
        tot = 0
        for op in wl.ops:
            if op["op"] == ("slice" if family == "slice" else "deform_slice"):
                C = op["src"][2]
                n = levels[op["level"]].n
                tot += m * 32 + n * C * u + m * C * 4 + (C * 4 if family == "deform_slice" else 0)
        return tot
    if family == "insert":
        per_level = m * 12 + m * (16 + 16 + 16)       # positions in, y / slots / weights out
        nlev = len(levels)
        return per_level + (nlev - 1) * (m * 16 + m * 48)
    return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--report", default=None, help="write a per-family timing report (JSON) here")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1912_05905_amd import lattice
    from paper_1912_05905_amd.pipeline import GpuPipeline
    from workloads import configs

    torch.cuda.set_device(0)
    lattice.lib()
    wl = configs.make(args.config)
    pipe = GpuPipeline(wl)
    stream = torch.cuda.current_stream()

    def one_step():
        levels, bufs, outs = pipe.step()
        return levels, bufs, outs

    # warmup (also sizes the pools)
    for _ in range(args.warmup):
        levels, _, _ = one_step()
        GpuPipeline.release(levels)
    torch.cuda.synchronize()

    # one instrumented step: per-family device time, to find the dominant family
    for f in FAMILIES:
        lattice.timing_enable(f, True)
    levels, _, _ = one_step()
    torch.cuda.synchronize()
    fam_ms = {f: lattice.timing_read(f) for f in FAMILIES}
    for f in FAMILIES:
        lattice.timing_enable(f, False)
    ns = {lv: levels[lv].n for lv in levels}
    flops = conv_flops(wl, levels)
    bytes_by_fam = {f: algorithmic_bytes(wl, levels, f) for f in FAMILIES}
    GpuPipeline.release(levels)
    dominant = max(fam_ms, key=lambda f: fam_ms[f][1])

    # timed region: K steps, dominant family timed with events on its stream
    lattice.timing_enable(dominant, True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        levels, _, _ = one_step()
        GpuPipeline.release(levels)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    launches, dom_ms = lattice.timing_read(dominant)
    lattice.timing_enable(dominant, False)

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = wl.m / (ms_per_step * 1e-3)
    dom_ms_step = dom_ms / args.steps
    dtype = "bf16" if wl.dtype == "bf16" else "f32"
    if dominant == "conv":
        peak = PEAK["mfma_bf16"] if dtype == "bf16" else PEAK["mfma_f32"]
        achieved = flops / (dom_ms_step * 1e-3)
        roof = {"bound": "mfma", "achieved": achieved / 1e12, "peak": peak / 1e12, "unit": "TFLOP/s",
                "frac": achieved / peak, "traffic": None}
    else:
        b = bytes_by_fam.get(dominant)
        achieved = (b / (dom_ms_step * 1e-3)) if b else None
        roof = {"bound": "hbm", "achieved": None if achieved is None else achieved / 1e9,
                "peak": PEAK["hbm"] / 1e9, "unit": "GB/s",
                "frac": None if achieved is None else achieved / PEAK["hbm"], "traffic": None}
    roof["kernel"] = dominant
    roof["launches_per_step"] = launches / args.steps
    roof["ms_per_step"] = dom_ms_step

    cpu = None
    if not args.no_cpu_baseline:
        from tests.oracle_pipeline import OraclePipeline
        c0 = time.perf_counter()
        OraclePipeline(wl).run()
        c1 = time.perf_counter()
        cpu = {"value": wl.m / (c1 - c0), "unit": "points/s", "cores": 1, "kind": "oracle",
               "sample": f"one full step of the same {wl.m}-point workload on the CPU oracle "
                         f"(std::map lattice, scalar float64), {c1 - c0:.1f} s"}

    line = {
        "metric": "points/s for splat+conv+slice at 120k pts; lattice-conv GFLOP/s (% MFMA peak)",
        "value": value, "unit": "points/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dtype, "data": "synthetic",
        "config": {"workload": f"config{wl.cfg}:{wl.name}", "points": wl.m,
                   "sigma": float(wl.sigma[0]), "vertices_per_level": [ns[k] for k in sorted(ns)],
                   "conv_gflop_per_step": flops / 1e9},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    if args.report:
        rep = {"families_ms_one_step": {f: fam_ms[f][1] for f in FAMILIES},
               "launches_one_step": {f: fam_ms[f][0] for f in FAMILIES},
               "bytes_per_step": bytes_by_fam, "conv_flops_per_step": flops,
               "ms_per_step": ms_per_step, "vertices": ns}
        with open(args.report, "w") as fh:
            json.dump(rep, fh, indent=1)


if __name__ == "__main__":
    main()
