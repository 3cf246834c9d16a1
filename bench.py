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
import gc
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"hbm": 8.0e12, "mfma_f32": 157.3e12, "mfma_bf16": 2.5e15}
BUILD_FAMILIES = {"fill", "insert", "scan", "lists", "nbr"}
FAMILIES = ["fill", "insert", "scan", "lists", "nbr", "splat", "distribute", "groupnorm", "conv", "slice",
            "deform_slice", "deform_bwd", "conv_bwd", "splat_bwd", "slice_bwd", "linear_bwd"]
# kernel symbol fragments of each family (rocprofv3 kernel names; first match
# wins).  Backward operators that reuse a forward kernel (the adjoint
# convolution on k_conv_lds, splat and slice as each other's adjoints, the
# finishing pass of the DeformSlice gradient gather) are only separable by
# the event timing, which names the outermost operator.
FAMILY_KERNELS = {
    "fill": ["k_clear_table"], "insert": ["k_insert_points"], "scan": ["k_scan("],
    "lists": ["k_fill_lists"], "nbr": ["k_level_tables", "k_mask_order"],
    "deform_bwd": ["k_deform_bwd", "DeformGradRows"],
    "conv_bwd": ["k_conv_wgrad", "k_wgrad_reduce", "k_conv_bwd_prep"], "linear_bwd": ["k_lin_"],
    "splat_bwd": ["k_scale_by_weight_sum"], "groupnorm": ["k_gn_"],
    "splat": ["k_splat_chunks", "k_splat_finish"], "distribute": ["k_dist_"], "conv": ["k_conv"],
    "slice": ["k_slice<"],
    "deform_slice": ["k_deform_slice", "k_deform_classify"],
}
CSRC = os.path.join(ROOT, "paper_1912_05905_amd", "csrc")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def kernel_source_hash() -> str:
    """Hash of the HIP sources: measured traffic is reported only while the
    kernels are the ones the counters were taken on."""
    import hashlib
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        with open(os.path.join(CSRC, name), "rb") as fh:
            h.update(name.encode() + fh.read())
    return h.hexdigest()[:16]


def family_of(kernel_name: str):
    for fam, frags in FAMILY_KERNELS.items():
        if any(f in kernel_name for f in frags):
            return fam
    return None


def default_layout(wl) -> tuple:
    """(pipelines, whether they share one build stream) that the bench runs
    by default, from timings of every workload on MI355X.  More clouds in
    flight help where one cloud's kernels (small levels, a few hundred
    workgroups) cannot fill the GPU: the 120k-point LiDAR workloads, and
    the 200k-point room with coarse levels, run three pipelines whose builds
    share one stream (four streams in all, one per hardware queue).  A
    training step runs two pipelines with a build stream each (three were
    slower), and so does the single-level 200k-point room, whose kernels
    are larger (three were slower there).  The 1M-point clouds run two
    pipelines on a shared build stream."""
    levels = 1 + sum(op["op"] == "coarsen" for op in wl.ops)
    if wl.grads:
        return 2, False
    if wl.m < 150_000 or (wl.m < 500_000 and levels > 1):
        return 3, True
    if wl.m < 500_000:
        return 2, False
    return 2, True


def default_pipelines(wl) -> int:
    return default_layout(wl)[0]


def summarize_pmc(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, copy_mb, steps, warmup, key, pipelines=2):
    """Per-family HBM bytes per step from rocprofv3 --pmc FETCH_SIZE and
    WRITE_SIZE runs of this benchmark, each counter scaled by what it reads
    for a device-to-device copy of copy_mb MiB.  Appends the result to
    profiles/traffic.json under `key`."""
    import csv
    import glob

    def counter_rows(d):
        files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        rows = []
        for f in files:
            rows += list(csv.DictReader(open(f)))
        return rows

    def per_kernel(rows, counter):
        out = {}
        for r in rows:
            if r.get("Counter_Name") != counter:
                continue
            out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return out

    def copy_value(d, counter):
        vals = per_kernel(counter_rows(d), counter)
        best = max(vals.items(), key=lambda kv: max(kv[1]))
        return max(best[1])

    nbytes = copy_mb * 2 ** 20
    scale_f = nbytes / copy_value(copy_fetch_dir, "FETCH_SIZE")
    scale_w = nbytes / copy_value(copy_write_dir, "WRITE_SIZE")
    fams = {}
    for d, counter, scale, field in ((fetch_dir, "FETCH_SIZE", scale_f, "fetch_bytes"),
                                      (write_dir, "WRITE_SIZE", scale_w, "write_bytes")):
        for name, vals in per_kernel(counter_rows(d), counter).items():
            fam = family_of(name)
            if fam is None:
                continue
            ent = fams.setdefault(fam, {"fetch_bytes": 0.0, "write_bytes": 0.0, "dispatches": 0})
            ent[field] += sum(vals) * scale
            if counter == "FETCH_SIZE":
                ent["dispatches"] += len(vals)
    runs = warmup + 1 + 2 * steps  # warmup, instrumented step, the two timed regions of the profiled run
    for fam, ent in fams.items():
        # each pipeline builds its next cloud's lattices one step ahead: one
        # more hierarchy per pipeline than steps
        n = runs + pipelines if fam in BUILD_FAMILIES else runs
        ent["fetch_bytes_per_step"] = ent.pop("fetch_bytes") / n
        ent["write_bytes_per_step"] = ent.pop("write_bytes") / n
        ent["dispatches_per_step"] = ent.pop("dispatches") / n
    data = json.load(open(TRAFFIC_FILE)) if os.path.exists(TRAFFIC_FILE) else {}
    stamp = os.path.join(fetch_dir, "source_hash.txt")
    if not os.path.exists(stamp):
        raise SystemExit(f"{stamp} missing: write it with bench.py --source-hash when the counters are taken")
    data[key] = {"kernel_source_hash": open(stamp).read().strip(), "fetch_scale": scale_f, "write_scale": scale_w,
                 "copy_mib": copy_mb, "families": fams}
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(data, fh, indent=1, sort_keys=True)
    print(json.dumps(data[key], indent=1))


def measured_traffic(key, family):
    """HBM bytes per step of a family from profiles/traffic.json, or None when
    absent or taken on different kernel sources."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    ent = json.load(open(TRAFFIC_FILE)).get(key)
    if not ent or ent.get("kernel_source_hash") != kernel_source_hash():
        return None
    fam = ent["families"].get(family)
    if not fam:
        return None
    return fam["fetch_bytes_per_step"] + fam["write_bytes_per_step"]


def conv_flops(wl, levels):
    """Nominal flops of all convolutions of one step: 2 * 9 * Cin * Cout per
    output vertex for the same-level and the strided (Downsample)
    convolution, and per coarse (input) vertex for Upsample, the transposed
    convolution, whose natural form multiplies every coarse vertex by the
    nine tap matrices."""
    total = 0
    for op in wl.ops:
        if op["op"] in ("conv", "conv_down"):
            total += 2 * levels[op["level"]].n * 9 * op["src"][2] * op["dst"][2]
        elif op["op"] == "refine":
            total += 2 * levels[op["level"] + 1].n * 9 * op["src"][2] * op["dst"][2]
    return total


def conv_bwd_flops(wl, levels):
    """Nominal flops of the convolution gradients of one step: dX and dW
    each cost what the forward convolution costs (counted as in
    conv_flops)."""
    total = 0
    for op in wl.ops:
        if op["op"] == "conv_bwd":
            cin, cout = op["x"][2], op["y"][2]
            lv = op["level"] + 1 if op["kind"] == "refine" else op["level"]
            total += 2 * 2 * levels[lv].n * 9 * cin * cout
    return total


def distribute_flops(wl):
    """Flops of the Distribute + PointNet layers of one step: each of the 4m
    (point, vertex) rows goes through the three 1x1 layers."""
    total = 0
    for op in wl.ops:
        if op["op"] == "distribute":
            k = 3 + wl.features.shape[1]
            for name in op["layers"]:
                W, _ = wl.mlp[name]
                total += 2 * 4 * wl.m * W.shape[0] * k
                k = W.shape[0]
    return total


def point_ops(wl, pipe):
    """The point-output operators of a step as they are launched: a slice
    followed by a DeformSlice of the same values runs as one fused pass."""
    fused = getattr(pipe, "_fused", set())
    out, skip = [], False
    for i, op in enumerate(wl.ops):
        if skip:
            skip = False
            continue
        if op["op"] in ("slice", "deform_slice"):
            if i in fused:
                out.append(("slice+deform", op))
                skip = True
            else:
                out.append((op["op"], op))
    return out


def algorithmic_bytes(wl, levels, family, pipe=None):
    """Bytes a kernel family must move per step (each input read once, each
    output written once), for the HBM-bound families."""
    u = 2 if wl.dtype == "bf16" else 4
    m = wl.m
    if family == "splat":
        C = next((op["dst"][2] for op in wl.ops if op["op"] == "splat"), None)
        if C is None:
            return None
        n = levels[0].n
        # features m*C*u, lists 4m*(4 entry + 4 weight), offsets, output n*C*u
        return m * C * u + 4 * m * 8 + (n + 1) * 4 + n * C * u
    if family in ("slice", "deform_slice"):
        # per point 32 B of vertex indices and weights and C*4 out per output,
        # the vertex rows n*C*u once; DeformSlice also reads wv.  The fused
        # slice + DeformSlice pass (timed as deform_slice) writes both rows.
        tot = 0
        for kind, op in point_ops(wl, pipe):
            fam = "slice" if kind == "slice" else "deform_slice"
            if fam != family:
                continue
            C = op["src"][2]
            n = levels[op["level"]].n
            outs = 2 if kind == "slice+deform" else 1
            tot += m * 32 + n * C * u + outs * m * C * 4 + (C * 4 if kind != "slice" else 0)
        return tot or None
    if family == "insert":
        # per level: positions in, elevated positions / slots / weights out
        # (the hierarchy call elevates the positions for every level; a level
        # coarsened on its own reads its parent's elevated positions instead)
        nlev = len(levels)
        coarse_in = 12 if pipe is not None and getattr(pipe, "_levels", 0) else 16
        return m * (12 + 48) + (nlev - 1) * m * (coarse_in + 48)
    return None


def conv_occupied_flops(wl, levels):
    """Flops of all convolutions of one step counted on the taps that exist:
    2 Cin Cout per (output vertex, tap) pair whose neighbour is allocated
    (a missing neighbour contributes nothing).  Waits for the device."""
    total = 0
    for op in wl.ops:
        lv = op.get("level")
        if op["op"] == "conv":
            pairs = levels[lv].conv_taps(levels[lv])
        elif op["op"] == "conv_down":
            pairs = levels[lv].conv_taps(levels[lv - 1])
        elif op["op"] == "refine":
            pairs = levels[lv].conv_taps(levels[lv + 1])
        else:
            continue
        total += 2 * pairs * op["src"][2] * op["dst"][2]
    return total


def host_cpu():
    """CPU model of this host and its logical CPU count."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model, os.cpu_count()


def _oracle_worker(args):
    """One process of the all-core CPU baseline: whole oracle steps of the
    workload for about `seconds`; returns (steps, seconds)."""
    cfg, seconds = args
    sys.path.insert(0, ROOT)
    from tests.oracle_pipeline import OraclePipeline
    from workloads import configs
    wl = configs.make(cfg)
    OraclePipeline(wl).run()           # first step untimed (library load, page-in)
    c0 = time.perf_counter()
    n = 0
    while True:
        OraclePipeline(wl).run()
        n += 1
        if time.perf_counter() - c0 >= seconds:
            break
    return n, time.perf_counter() - c0


def cpu_baseline(wl, seconds=10.0, workers=None):
    """The CPU oracle on this host: one thread (whole steps for about
    `seconds`, with per-operation times), then all cores (one process per
    core, each running whole steps for about `seconds`)."""
    from concurrent.futures import ProcessPoolExecutor
    import multiprocessing as mp
    from tests.oracle_pipeline import OraclePipeline
    model, ncpu = host_cpu()
    times = {}
    c0 = time.perf_counter()
    nsteps = 0
    while True:
        OraclePipeline(wl).run(times=times)
        nsteps += 1
        if time.perf_counter() - c0 >= seconds or nsteps >= 50:
            break
    t1 = time.perf_counter() - c0
    one = nsteps * wl.m / t1
    # GPU machines give a process a share of 16 cores whatever nproc says
    workers = workers or max(1, min(ncpu or 1, 16))
    with ProcessPoolExecutor(max_workers=workers, mp_context=mp.get_context("spawn")) as ex:
        res = list(ex.map(_oracle_worker, [(wl.cfg, seconds)] * workers))
    allc = sum(n * wl.m / t for n, t in res)
    return {"value": allc, "unit": "points/s", "cores": workers, "kind": "oracle",
            "sample": f"whole steps of the same {wl.m}-point workload on the CPU oracle (std::map lattice, scalar "
                      f"float64): {workers} processes, one per core, each for about {seconds:.0f} s "
                      f"({sum(n for n, _ in res)} steps in all); single thread {nsteps} steps in {t1:.1f} s",
            "cpu_model": model, "nproc": ncpu, "value_1thread": one,
            "ms_per_step_1thread": t1 * 1e3 / nsteps,
            "op_ms_1thread": {k: v * 1e3 / nsteps for k, v in times.items()}}


def _hbm_entry(nbytes, ms):
    if not nbytes or not ms:
        return None
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"algorithmic_bytes": nbytes, "ms_per_step": ms, "achieved_GBps": gbs, "frac": gbs * 1e9 / PEAK["hbm"]}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--streams", type=int, default=0,
                    help="pipelines (each with a compute stream) that take the clouds in turn; 0: automatic")
    ap.add_argument("--build", choices=("auto", "own", "shared"), default="auto",
                    help="a build stream per pipeline (own) or one for all (shared); auto: as --streams 0")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="seconds of oracle work per CPU-baseline leg")
    ap.add_argument("--report", default=None, help="write a per-family timing report (JSON) here")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run device-to-device copies of MIB MiB (PMC scale calibration)")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR"),
                    help="summarise rocprofv3 --pmc runs into profiles/traffic.json")
    ap.add_argument("--copy-mib", type=int, default=256)
    ap.add_argument("--source-hash", action="store_true", help="print the hash of the HIP sources and exit")
    args = ap.parse_args()
    if args.source_hash:
        print(kernel_source_hash())
        return
    if args.summarize_pmc:
        from workloads import configs
        pipelines = args.streams or default_pipelines(configs.make(args.config))
        summarize_pmc(*args.summarize_pmc, args.copy_mib, args.steps, args.warmup, f"config{args.config}",
                      pipelines)
        return
    if args.calibrate_copy:
        import torch
        src = torch.ones(args.calibrate_copy * 2 ** 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"copied {args.calibrate_copy} MiB x3", flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import statistics

    import torch

    from paper_1912_05905_amd import lattice
    from paper_1912_05905_amd.pipeline import GpuPipeline
    from workloads import configs

    torch.cuda.set_device(0)
    lattice.lib()
    wl = configs.make(args.config)
    # Consecutive steps overlap.  `streams` pipelines take the clouds in
    # turn, each with buffers of its own: a pipeline builds its next cloud's
    # lattices one step ahead on a build stream (its own, or one the
    # pipelines share) and runs its operators on its compute stream (the
    # first one on the current stream), so that the small coarse levels'
    # kernels (a few hundred workgroups each) and the latency-bound build
    # chains share the GPU.  The layouts use at most four streams, one per
    # hardware queue of the HIP runtime's default; a fifth stream would share
    # a queue with another and serialise behind it.  Every step still does
    # all of its work.
    if args.streams < 0:
        print("--streams must be 0 (automatic) or at least 1", file=sys.stderr)
        sys.exit(2)
    layout = default_layout(wl)
    if args.streams == 0:
        args.streams = layout[0]
    shared = layout[1] if args.build == "auto" else args.build == "shared"
    build_stream = torch.cuda.Stream() if shared and args.streams > 1 else None
    pipes = [GpuPipeline(wl, overlap=True, build_stream=build_stream) for _ in range(args.streams)]
    streams = [torch.cuda.current_stream()] + [torch.cuda.Stream() for _ in range(args.streams - 1)]
    issued = [0]   # steps issued so far: step g runs on pipeline / stream g % streams

    def one_step():
        k = issued[0] % args.streams
        issued[0] += 1
        if args.streams > 1:
            torch.cuda.set_stream(streams[k])   # (cheaper than a stream context per step)
        levels, bufs, outs = pipes[k].step()
        pipes[k].finish_step(levels)
        return levels, bufs, outs

    def last_stream():
        return streams[(issued[0] - 1) % args.streams]

    # warmup (also sizes the pools)
    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()

    # one instrumented step: per-family device time, to find the dominant
    # family; the tap occupancy of its convolutions
    for f in FAMILIES:
        lattice.timing_enable(f, True)
    levels, _, _ = one_step()
    inst = pipes[(issued[0] - 1) % args.streams]
    torch.cuda.synchronize()
    fam_ms = {f: lattice.timing_read(f) for f in FAMILIES}
    for f in FAMILIES:
        lattice.timing_enable(f, False)
    ns = {lv: levels[lv].n for lv in levels}
    flops = conv_flops(wl, levels)
    occ_flops = conv_occupied_flops(wl, levels) if flops else 0
    bwd_flops = conv_bwd_flops(wl, levels)
    bytes_by_fam = {f: algorithmic_bytes(wl, levels, f, inst) for f in FAMILIES}
    torch.cuda.synchronize()
    dominant = max(fam_ms, key=lambda f: fam_ms[f][1])

    # timed region: K steps, nothing instrumented; every `win` steps an
    # event on the stream of the step issued last gives per-window device
    # throughput (median reported)
    win = max(1, args.steps // 20)
    marks = []
    # Python's cyclic garbage collector is kept out of the timed regions (as
    # timeit does): a full collection over the interpreter's objects (torch
    # included) stalls the issuing thread for tens of milliseconds, which
    # landed in some runs' timed region as +50% on the mean step time
    gc.collect()
    gc.freeze()
    gc.disable()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        if i % win == 0:
            ev = torch.cuda.Event(enable_timing=True)
            ev.record(last_stream())
            marks.append((i, ev))
        one_step()
    end = torch.cuda.Event(enable_timing=True)
    end.record(last_stream())
    marks.append((args.steps, end))
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    windows = [marks[j][1].elapsed_time(marks[j + 1][1]) / (marks[j + 1][0] - marks[j][0])
               for j in range(len(marks) - 1)]

    # the same K steps again with the kernels of the dominant family and of
    # the HBM-bound operators timed: each launch's start / stop HIP events
    # are bound to its dispatch on the stream it runs on, so a family's sum
    # is its kernel time; these completion events delay the next kernel, so
    # this region's wall time is reported beside the first, not as the
    # throughput
    timed = [dominant] + [f for f in ("splat", "slice", "deform_slice", "insert")
                          if f != dominant and bytes_by_fam.get(f)]
    for f in timed:
        lattice.timing_enable(f, True)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(args.steps):
        one_step()
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    gc.enable()
    gc.unfreeze()
    fam_timed = {f: lattice.timing_read(f) for f in timed}
    for f in timed:
        lattice.timing_enable(f, False)
    for p in pipes:
        p.flush()
    launches, dom_ms = fam_timed[dominant]

    # the dominant family once more on one pipeline (its launches beside the
    # next cloud's build only), for the kernels' position without the other
    # clouds' operators beside them; not part of the throughput
    one_ms = None
    if args.streams > 1:
        solo = GpuPipeline(wl, overlap=True)
        n_solo = min(args.steps, 100)
        for _ in range(5):
            levels_s, _, _ = solo.step()
            solo.finish_step(levels_s)
        torch.cuda.synchronize()
        lattice.timing_enable(dominant, True)
        for _ in range(n_solo):
            levels_s, _, _ = solo.step()
            solo.finish_step(levels_s)
        torch.cuda.synchronize()
        solo_launches, solo_ms = lattice.timing_read(dominant)
        lattice.timing_enable(dominant, False)
        solo.flush()
        one_ms = solo_ms / n_solo

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = wl.m / (ms_per_step * 1e-3)
    dom_ms_step = dom_ms / args.steps
    dtype = "bf16" if wl.dtype == "bf16" else "f32"
    mfma_flops = {"conv": flops, "distribute": distribute_flops(wl), "conv_bwd": bwd_flops}
    if dominant in mfma_flops:
        peak = PEAK["mfma_bf16"] if dtype == "bf16" else PEAK["mfma_f32"]
        achieved = mfma_flops[dominant] / (dom_ms_step * 1e-3)
        roof = {"bound": "mfma", "achieved": achieved / 1e12, "peak": peak / 1e12, "unit": "TFLOP/s",
                "frac": achieved / peak, "traffic": None}
        if dominant == "conv" and occ_flops:
            # the same launches counted on the taps that exist
            occ = occ_flops / (dom_ms_step * 1e-3)
            roof["flops_definition"] = ("nominal: 2*9*Cin*Cout per output vertex (per coarse vertex for "
                                        "Upsample); occupied: 2*Cin*Cout per (vertex, tap) pair whose "
                                        "neighbour exists")
            roof["gflop_per_step_nominal"] = flops / 1e9
            roof["gflop_per_step_occupied"] = occ_flops / 1e9
            roof["occupied_tap_fraction"] = occ_flops / flops
            roof["achieved_occupied"] = occ / 1e12
            roof["frac_occupied"] = occ / peak
        if one_ms:
            roof["one_pipeline"] = {"ms_per_step": one_ms, "frac": mfma_flops[dominant] / (one_ms * 1e-3) / peak}
            if dominant == "conv" and occ_flops:
                roof["one_pipeline"]["frac_occupied"] = occ_flops / (one_ms * 1e-3) / peak
    else:
        b = bytes_by_fam.get(dominant)
        achieved = (b / (dom_ms_step * 1e-3)) if b else None
        roof = {"bound": "hbm", "achieved": None if achieved is None else achieved / 1e9,
                "peak": PEAK["hbm"] / 1e9, "unit": "GB/s",
                "frac": None if achieved is None else achieved / PEAK["hbm"], "traffic": None}
    t = measured_traffic(f"config{wl.cfg}", dominant)
    if t is not None:
        roof["traffic"] = t / max(launches / args.steps, 1)
    roof["kernel"] = dominant
    roof["launches_per_step"] = launches / args.steps
    roof["ms_per_step"] = dom_ms_step
    roof["ms_per_launch"] = dom_ms / max(launches, 1)
    roof["timed_region_ms_per_step"] = (t3 - t2) * 1e3 / args.steps
    roof["launch_context"] = (f"durations of launches that share the GPU with the other {args.streams - 1} "
                              "pipeline(s)' operators and with the lattice builds, as the step runs them"
                              if args.streams > 1 else "durations of launches beside the next cloud's build")
    # the HBM-bound operators, each over its own launches in the same region
    hbm = {}
    for f in timed:
        if f == dominant:
            continue
        e = _hbm_entry(bytes_by_fam.get(f), fam_timed[f][1] / args.steps)
        if e:
            tr = measured_traffic(f"config{wl.cfg}", f)
            e["traffic_bytes_per_step"] = tr
            hbm[f] = e
    roof["hbm_families"] = hbm

    cpu = None if args.no_cpu_baseline else cpu_baseline(wl, args.cpu_seconds)

    line = {
        "metric": "points/s for splat+conv+slice at 120k pts; lattice-conv GFLOP/s (% MFMA peak)",
        "value": value, "unit": "points/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dtype, "data": "synthetic",
        "config": {"workload": f"config{wl.cfg}:{wl.name}", "points": wl.m,
                   "sigma": float(wl.sigma[0]), "vertices_per_level": [ns[k] for k in sorted(ns)],
                   "conv_gflop_per_step": flops / 1e9,
                   "conv_gflop_per_step_occupied_taps": occ_flops / 1e9,
                   "distribute_gflop_per_step": mfma_flops["distribute"] / 1e9,
                   "conv_bwd_gflop_per_step": bwd_flops / 1e9,
                   "pipelines": args.streams,
                   "build_streams": 1 if build_stream is not None else args.streams,
                   "steps_overlap": "pipelines take the clouds in turn, each building its next cloud's "
                                    "lattices one step ahead on a build stream while its operators run on "
                                    "its own compute stream; every step does all of its work"},
        "timing": {"timed_ms": (t1 - t0) * 1e3, "windows": len(windows), "steps_per_window": win,
                   "ms_per_step_median_window": statistics.median(windows),
                   "ms_per_step_min_window": min(windows), "ms_per_step_max_window": max(windows),
                   "python_gc": "collected and frozen before the timed regions, disabled during them"},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    if args.report:
        rep = {"families_ms_one_step": {f: fam_ms[f][1] for f in FAMILIES},
               "launches_one_step": {f: fam_ms[f][0] for f in FAMILIES},
               "bytes_per_step": bytes_by_fam, "conv_flops_per_step": flops,
               "conv_flops_per_step_occupied": occ_flops,
               "ms_per_step": ms_per_step, "vertices": ns}
        with open(args.report, "w") as fh:
            json.dump(rep, fh, indent=1)


if __name__ == "__main__":
    main()
