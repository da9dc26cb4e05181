#!/usr/bin/env python3
"""Throughput of the sparsity-preserved LoRA linear (forward + backward) on one GPU.

One step = lors_forward + lors_backward over one batch of seeded synthetic
inputs already resident in HBM (every step of the layer runs in liblors.so;
mask preparation -- packing and the transposed layout the backward reads --
happens once per layer, before timing, since the mask is frozen).  With
--graph the step is captured once as a HIP graph and replayed (a replay must
reproduce the eager step first); by default the library calls are issued from
Python every step.

Before the W warm-up steps the step runs untimed for --settle-s seconds: an
idle GPU needs on the order of 100 ms of sustained load to reach its working
clock, so a timed window right after start-up would measure that ramp rather
than a training loop's steady state.

Prints ONE JSON line: whole-job TFLOP/s over the algorithmic flops
6RCL + 8rRC per step, the fraction of the bf16 MFMA peak, peak bytes, the
roofline entry of the dominant kernel (HIP-event durations on the launch
stream) and the fp64 CPU oracle timed on the host's cores.  The default
workload is the largest single-GPU projection, Llama-3-8B down_proj
(4096 x 14336, 8192 tokens, r = 64, 70 % magnitude mask); the two
Llama-2-7B projections (q_proj 4096 x 4096; up_proj 11008 x 4096 with a 2:4
mask) are timed in the same run and reported under "other_workloads"
(--also '' turns that off).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "masked-LoRA linear fwd+bwd TFLOP/s (bf16) and % of MFMA peak; peak bytes"
DEFAULT_WORKLOAD = "llama3_8b_down_proj"
DEFAULT_ALSO = "llama2_7b_q_proj,llama2_7b_up_proj_2_4"
# MI355X dense MFMA peaks in TFLOP/s: 256 CUs x 4 matrix cores x 2.4 GHz x
# (1024 bf16 or 256 fp32 flops per clock per matrix core).  HBM3E 8 TB/s.
PEAK_TFLOPS = {"bf16": 2516.6, "f32": 157.3}
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--settle-s", type=float, default=1.0,
                    help="seconds of untimed steps before the warm-up (the GPU leaves its idle clocks)")
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--also", default=DEFAULT_ALSO,
                    help="comma-separated workloads whose step is also timed (same settling, warm-up and step "
                         "count) and reported under other_workloads; '' for none")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle timing (profiling runs)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="minimum host time spent on the oracle sample")
    ap.add_argument("--ste", action="store_true",
                    help="straight-through adapter gradients (Section 2.3) in the weight half; "
                         "flops counted are those of that method")
    ap.add_argument("--sparse-mfma", action="store_true",
                    help="2:4 workloads: forward on the structured-sparse MFMA")
    ap.add_argument("--graph", action="store_true",
                    help="replay one captured HIP graph of the step instead of issuing the library calls "
                         "from Python every step (per-kernel timings are eager either way)")
    ap.add_argument("--pmc-probe", action="store_true",
                    help="short program for hardware-counter runs: one step, a device copy of "
                         "COPY_BYTES (the calibration of the byte counters), one more step")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="no GPU work: print the HBM-traffic summary of --workload from the counter CSVs of two "
                         "rocprofv3 --pmc runs of --pmc-probe (FETCH_SIZE, then WRITE_SIZE)")
    return ap.parse_args()


COPY_BYTES = 256 << 20

# Sources that define each timed kernel: a traffic figure measured with
# hardware counters is reported only while these files are unchanged.
KERNEL_SOURCES = {
    "fwd_kernel": ["fwd_bf16.hip"],
    "dx_kernel": ["dx_bf16.hip"],
    "g_kernel": ["g_bf16.hip"],
}
COMMON_SOURCES = ["gemm_common.hpp", "device_common.hpp", "kernels.hpp"]


def kernel_digest(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel] + COMMON_SOURCES:
        with open(os.path.join(ROOT, "paper_2501_08582_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` from profiles/traffic_<workload>.txt
    (rocprofv3 FETCH_SIZE / WRITE_SIZE, calibrated on a copy of known size),
    or None when absent or taken on different kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")
    if kernel is None or not os.path.exists(path):
        return None
    for line in open(path):
        f = line.split()
        if len(f) == 5 and f[0] == kernel:
            return int(f[3]) if f[4] == kernel_digest(kernel) else None
    return None


def traffic_summary(workload: str, fetch_csv: str, write_csv: str, commands=()) -> str:
    """The profiles/traffic_<workload>.txt text from the counter CSVs of two
    --pmc-probe runs.  Each counter is calibrated on the probe's device copy of
    COPY_BYTES (read and written once each); a kernel's figure is the mean of
    its last two dispatches, the probe's two steps (a dX launch at set-up,
    which writes the transposed mask, comes before them)."""
    import csv

    def per_kernel(path, counter):
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        # the calibration copy is the probe's large one (mask preparation may
        # add small copies of its own, e.g. the 2:4 validity flag)
        copy = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        copy = [max(copy)] if copy else []
        if not copy or copy[0] * 1024 < COPY_BYTES / 4:
            raise ValueError(f"{path}: no calibration copy of {COPY_BYTES} bytes found")
        vals = {}
        for k in KERNEL_SOURCES:
            v = [float(r["Counter_Value"]) for r in rows if f"::{k}<" in r["Kernel_Name"]]
            if len(v) >= 2:
                vals[k] = sum(v[-2:]) / 2
        return copy[0], vals

    cf, fetch = per_kernel(fetch_csv, "FETCH_SIZE")
    cw, write = per_kernel(write_csv, "WRITE_SIZE")
    ff, fw = COPY_BYTES / (cf * 1024), COPY_BYTES / (cw * 1024)
    lines = [f"# HBM traffic per launch, {workload} (one layer step, bf16)",
             "# Commands (repository root, TMPDIR=/tmp), one counter per run:"]
    lines += [f"#   {c}" for c in commands]
    lines += [f"# Calibration: the {COPY_BYTES}-byte device copy (__amd_rocclr_copyBuffer) reads",
              f"#   FETCH_SIZE {cf:.1f} KiB and WRITE_SIZE {cw:.1f} KiB,",
              f"#   so traffic = FETCH_SIZE * 1024 * {ff:.5f} + WRITE_SIZE * 1024 * {fw:.5f} bytes.",
              "# Values are the mean of each kernel's last two dispatches (the probe run's two steps).",
              "# kernel  fetch_KiB  write_KiB  traffic_bytes  source_digest"]
    for k in KERNEL_SOURCES:
        if k in fetch and k in write:
            t = int(round(fetch[k] * 1024 * ff + write[k] * 1024 * fw))
            lines.append(f"{k} {fetch[k]:.1f} {write[k]:.1f} {t} {kernel_digest(k)}")
    return "\n".join(lines) + "\n"


def cpu_baseline(inp, args):
    """The fp64 oracle on the same workload, timed on the host cores."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import bf16 as obf16
    from oracle import lors as olors
    from paper_2501_08582_amd import costs

    wl = inp.wl
    f = obf16.to_f64 if wl.dtype == "bf16" else (lambda a: np.asarray(a, dtype=np.float64))
    # Bounded sample: one full forward+backward of the layer, repeated until
    # --cpu-seconds have passed (best pass reported).
    Ls = wl.L
    X, dY = f(inp.X[:Ls]), f(inp.dY[:Ls])
    W, B, A = f(inp.W), f(inp.B), f(inp.A)
    best, n, t_all = None, 0, time.perf_counter()
    while True:
        t0 = time.perf_counter()
        olors.forward(X, W, inp.M, B, A, wl.scale)
        olors.backward(dY, X, W, inp.M, B, A, wl.scale)
        dt = time.perf_counter() - t0
        best = dt if best is None else min(best, dt)
        n += 1
        if time.perf_counter() - t_all >= args.cpu_seconds or n >= 20:
            break
    flops = costs.algorithmic_flops(wl.R, wl.C, Ls, wl.r)
    threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"]
                  or [1])
    cpu_model = next((ln.split(":", 1)[1].strip() for ln in open("/proc/cpuinfo")
                      if ln.startswith("model name")), "unknown") if os.path.exists("/proc/cpuinfo") else "unknown"
    blas = next((f"{p.get('internal_api')} {p.get('version')}" for p in threadpool_info()
                 if p.get("user_api") == "blas"), "unknown")
    return {
        "value": flops / best / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "cpu_model": cpu_model,
        "blas": f"numpy {np.__version__}, {blas}",
        "kind": "oracle",
        "sample": (f"{wl.name}: {wl.R}x{wl.C} weight, r={wl.r}, {Ls} of {wl.L} tokens; "
                   f"numpy fp64 forward+backward, best of {n} passes ({best:.2f} s each)"),
    }


def main():
    args = parse()
    if args.traffic_from:
        cmds = [f"rocprofv3 --pmc {c} --output-format csv -d {os.path.dirname(f)} -o pmc "
                f"-- python -u bench.py --pmc-probe --workload {args.workload}"
                for c, f in zip(("FETCH_SIZE", "WRITE_SIZE"), args.traffic_from)]
        cmds.append(f"python bench.py --workload {args.workload} --traffic-from {' '.join(args.traffic_from)}")
        sys.stdout.write(traffic_summary(args.workload, *args.traffic_from, commands=cmds))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the layer shards by tokens, see the design notes)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2501_08582_amd import costs, synth
    from paper_2501_08582_amd.step import LayerStep

    wl = synth.workload(args.workload)
    inp = synth.make(wl)
    dt = wl.dtype
    R, C, L, r, s = wl.R, wl.C, wl.L, wl.r, wl.scale
    torch.cuda.set_device(0)
    layer = LayerStep(inp, ste=args.ste, sparse_mfma=args.sparse_mfma)
    ws = layer.ws
    stream = torch.cuda.current_stream()

    def step():
        layer.run()

    if args.pmc_probe:
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        step()
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        step()
        torch.cuda.synchronize()
        print(json.dumps({"pmc_probe": True, "workload": wl.name, "copy_bytes": COPY_BYTES}), flush=True)
        return

    t_settle = time.perf_counter()
    while time.perf_counter() - t_settle < args.settle_s:
        for _ in range(20):
            step()
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    launch = "eager"
    if args.graph:
        # One step captured as a HIP graph (the library allocates nothing and
        # records no memset), replayed K times; a replay must reproduce the
        # eager step's outputs before anything is timed.
        outs = (layer.Y, layer.dX, layer.dB, layer.dA)
        ref = [t.clone() for t in outs]
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step()
        stream.wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            step()
        for t in outs:
            t.zero_()
        graph.replay()
        torch.cuda.synchronize()
        exact = all(torch.equal(a, b) for a, b in zip(outs[:2], ref[:2]))
        close = all(float((a.double() - b.double()).norm()) <= 1e-5 * float(b.double().norm()) + 1e-30
                    for a, b in zip(outs[2:], ref[2:]))  # fp32 atomics: summation order varies
        if not (exact and close):
            print("bench.py: the graph replay does not reproduce the eager step", file=sys.stderr)
            sys.exit(1)
        step = graph.replay  # noqa: F811
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        launch = "hip graph replay"

    # Timed region: K steps bracketed by a device synchronisation on both
    # sides, HIP events on the launch stream at its two ends only.
    torch.cuda.reset_peak_memory_stats()
    mem0 = torch.cuda.memory_allocated()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        step()
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    transient = torch.cuda.max_memory_allocated() - mem0
    ms_total = start.elapsed_time(end)
    ms_step = ms_total / args.steps

    # Per-kernel durations inside the step: K more steps, each issued as its
    # three calls -- the forward, the data half (the dX kernel alone, the
    # transposed mask being built already) and the weight half (the dA/dB
    # clear plus the G kernel) -- with an event on the launch stream before,
    # between and after them.  Timing the calls in the step's own order
    # keeps each kernel's cache state that of the training loop: a kernel
    # repeated back to back finds much of its operands in the GPU's last-level
    # cache and runs faster than it does after the others.  The markers cost a
    # few microseconds, so the headline value above comes from the unmarked
    # steps; these marked steps also give the per-step spread.
    def marked_step(ev):
        ev[0].record(stream)
        layer.forward()
        ev[1].record(stream)
        layer.backward_data(reuse_mask_t=True)
        ev[2].record(stream)
        layer.backward_weight()
        ev[3].record(stream)

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for ev in evs:
        marked_step(ev)
    torch.cuda.synchronize()
    per_step_us = sorted(ev[0].elapsed_time(ev[3]) * 1e3 for ev in evs)
    avg = {k: sum(ev[i].elapsed_time(ev[i + 1]) for ev in evs) / len(evs)
           for i, k in enumerate(("fwd", "bwd_data", "bwd_weight"))}
    kflops = {"fwd": costs.fwd_flops(R, C, L, r), "bwd_data": costs.dx_flops(R, C, L, r),
              "bwd_weight": costs.ste_weight_flops(R, C, L, r) if args.ste else costs.g_flops(R, C, L, r)}
    kbytes = costs.min_hbm_bytes(R, C, L, r, elt=2 if dt == "bf16" else 4)
    kbytes = {"fwd": kbytes["fwd"], "bwd_data": kbytes["dx"], "bwd_weight": kbytes["g"]}
    kernel_names = {"fwd": "fwd_kernel", "bwd_data": "dx_kernel",
                    "bwd_weight": ("straight-through kernels (+ dA/dB clear)" if args.ste
                                   else "g_kernel (+ dA/dB clear)")}
    kernel_ids = {"fwd": "fwd_kernel", "bwd_data": "dx_kernel", "bwd_weight": None if args.ste else "g_kernel"}

    flops = costs.ste_step_flops(R, C, L, r) if args.ste else costs.algorithmic_flops(R, C, L, r)
    value = flops / (ms_step * 1e-3) / 1e12
    # executed: every 256-token tile of the forward and dX re-merges its W' tile
    executed = costs.executed_flops(R, C, L, r, 256, 256)
    if args.ste:
        executed += costs.ste_weight_flops(R, C, L, r) - costs.g_flops(R, C, L, r)
    peak = PEAK_TFLOPS[dt]
    dom = max(avg, key=avg.get)
    achieved = kflops[dom] / (avg[dom] * 1e-3) / 1e12
    elt = 2 if dt == "bf16" else 4
    traffic = measured_traffic(wl.name, kernel_ids[dom])
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dt,
        "data": "synthetic (seeded, Llama-shaped; random-init weights and adapters)",
        "config": {"workload": wl.name, "R": R, "C": C, "L": L, "r": r, "mask": wl.mask,
                   "sparsity": wl.sparsity, "scale": s,
                   "weight_gradient": "straight-through" if args.ste else "exact masked",
                   "forward_mfma": "structured-sparse" if args.sparse_mfma else "dense",
                   "step_launch": launch, "settle_s": args.settle_s,
                   "mask_prep": "packed mask and its transpose built once per layer, before timing"},
        "pct_mfma_peak": round(100.0 * value / peak, 2),
        "executed_tflops": round(executed / (ms_step * 1e-3) / 1e12, 2),
        "step_us_marked": {"median": round(per_step_us[len(per_step_us) // 2], 1),
                           "min": round(per_step_us[0], 1),
                           "calls": "forward | data half (dX) | weight half (dA/dB clear + G)"},
        "peak_bytes": {
            "weight_buffers": costs.weight_buffer_bytes(R, C, r, elt),
            "saved_activation": costs.saved_activation_bytes(C, L, elt),
            "workspace": ws,
            "transient_during_fwd_bwd": int(transient),
            "merged_weight_would_be": elt * R * C,
        },
        "kernels": {k: {"ms": round(avg[k], 4), "tflops": round(kflops[k] / (avg[k] * 1e-3) / 1e12, 1),
                        "pct_peak": round(100 * kflops[k] / (avg[k] * 1e-3) / 1e12 / peak, 2)}
                    for k in avg},
        "roofline": {
            "kernel": kernel_names[dom],
            "bound": "mfma",
            "achieved": round(achieved, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": traffic,
            "traffic_gbs": round(traffic / (avg[dom] * 1e-3) / 1e9, 1) if traffic else None,
            "algorithmic_bytes": kbytes[dom],
        },
        "wall_s_timed": round(wall, 4),
    }
    others = [w for w in args.also.split(",") if w and w != wl.name] if not (args.graph or args.pmc_probe) else []
    if others:
        del layer
        torch.cuda.empty_cache()
        out["other_workloads"] = [time_other(w, args) for w in others]
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(inp, args)
    print(json.dumps(out), flush=True)


def time_other(name, args):
    """Step time of another workload, measured like the headline (settling,
    warm-up, K steps between two events on the launch stream)."""
    import torch

    from paper_2501_08582_amd import costs, synth
    from paper_2501_08582_amd.step import LayerStep

    wl = synth.workload(name)
    layer = LayerStep(synth.make(wl), ste=args.ste, sparse_mfma=args.sparse_mfma)
    stream = torch.cuda.current_stream()
    t_settle = time.perf_counter()
    while time.perf_counter() - t_settle < args.settle_s:
        for _ in range(20):
            layer.run()
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        layer.run()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        layer.run()
    end.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    R, C, L, r = wl.R, wl.C, wl.L, wl.r
    flops = costs.ste_step_flops(R, C, L, r) if args.ste else costs.algorithmic_flops(R, C, L, r)
    tf = flops / (ms * 1e-3) / 1e12
    del layer
    torch.cuda.empty_cache()
    return {"workload": name, "R": R, "C": C, "L": L, "r": r, "mask": wl.mask, "ms_per_step": round(ms, 4),
            "tflops": round(tf, 2), "pct_mfma_peak": round(100.0 * tf / PEAK_TFLOPS[wl.dtype], 2)}


if __name__ == "__main__":
    main()
