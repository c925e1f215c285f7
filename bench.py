"""Benchmark of the fused selective scan forward on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu]

One step is one call of the fused selective scan (every step of the hot path:
exp discretisation, the recurrence, the C contraction, the D skip and the
h_last write; bf16 widening on the bf16 workload) over one batch of synthetic
input that is already resident in HBM.  The default workload is the largest
single-GPU one, B=1, D=5120, N=16, L=65536 in fp32 (4.04 GB of algorithmic
traffic per step).  Several input sets are rotated so that the working set is
larger than the 256 MB MALL and each step streams its inputs from HBM.

Prints one JSON line: throughput in B*L*D*N elements/s over exactly K timed
steps run back to back after W untimed ones (preceded by a clock warm-up of
at least --clock-warmup-ms of launches, stated in the line), the HBM roofline
of the call (algorithmic bytes / mean call duration, the interval between HIP
events recorded on the launch stream around the K steps divided by K, against
8 TB/s; the spread of single calls from an untimed pass afterwards), its fp32
arithmetic against the fp32 vector peak, and the CPU oracle timed on the host
cores over a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads as wl  # noqa: E402

DEFAULT_WORKLOAD = "selective_f32_b1_d5120_n16_l65536"

# MI355X figures used for the roofline
HBM_PEAK_GBS = 8000.0            # HBM3E, 8 TB/s
N_CU, SIMD_PER_CU, CLOCK_HZ = 256, 4, 2.4e9
# fp32 vector peak, as published: 157.3 TFLOP/s
FP32_PEAK_TFLOPS = 157.3
# fp32 flops the method does per (b,d,t,n) element: delta*A' (1), (delta*x)*B
# (1), the state FMA (2), the C FMA (2); the exp2 is not a flop and is not counted
FLOP_PER_ELEM = 6.0
FLOP_PER_ELEM_BWD = 14.0
MALL_BYTES = 256 << 20


def algorithmic_bytes(w) -> int:
    """Each input read once, each output written once (fp32 y and h_last)."""
    es = 2 if w.dtype == "bf16" else 4
    x_dl = 2 * w.B * w.D * w.L * es
    bc = 2 * w.B * w.L * w.N * es
    a_d = w.D * w.N * 4 + w.D * 4
    out = w.B * w.D * w.L * 4 + w.B * w.D * w.N * 4
    return x_dl + bc + a_d + out


# the sources each path's kernels are built from (traffic records are keyed to them)
FWD_SOURCES = ("selective_common.h", "selective_scan.hip", "selective_scan16.hip",
               "selective_scan_quad.hip", "sw_internal.h")
AFFINE_SOURCES = ("affine_scan.hip", "sw_internal.h")
BWD_SOURCES = ("selective_bwd.hip", "selective_common.h", "sw_internal.h")

# workload -> committed HBM traffic record (rocprofv3 FETCH_SIZE / WRITE_SIZE)
TRAFFIC_RECORDS = {
    "selective_f32_b1_d5120_n16_l65536": "selective_quad_f32_b1_d5120_n16_l65536_traffic.txt",
    "selective_f32_b4_d2048_n16_l8192_stress":
        "selective_row16_f32_b4_d2048_n16_l8192_stress_traffic.txt",
    "selective_bf16_b8_d1536_n16_l2048": "selective_row16_bf16_b8_d1536_n16_l2048_traffic.txt",
    "affine_f32_b1_d5120_l65536": "affine_rows_f32_b1_d5120_l65536_traffic.txt",
    "affine_f32_b8_d1536_l2048": "affine_scan_f32_b8_d1536_l2048_traffic.txt",
}
# the backward given the forward's checkpoints (no Mamba-block options)
BWD_TRAFFIC_RECORDS = {
    "selective_bf16_b8_d1536_n16_l2048": "selective_bwd_bf16_b8_d1536_n16_l2048_ckpt_traffic.txt",
}


def kernel_source_sha256(path: str = "selective") -> str:
    """Hash of the sources and headers of one path's kernels (sorted by name)."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_00601_amd", "csrc")
    names = {"affine": AFFINE_SOURCES, "bwd": BWD_SOURCES}.get(path, FWD_SOURCES)
    for p in sorted(os.path.join(csrc, f) for f in names):
        h.update(os.path.basename(p).encode())
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(w, launch=None, bwd=False):
    """HBM bytes per call from the committed counter summary, if it was taken on
    the current kernel sources, this workload and (for the fused forward) the
    same launches; else None.  bwd: the backward's record."""
    name = (BWD_TRAFFIC_RECORDS if bwd else TRAFFIC_RECORDS).get(w.name)
    if name is None:
        return None
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    sha = kernel_source_sha256("bwd" if bwd else w.path)
    rec = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                rec[k.strip()] = v.strip()
    if rec.get("kernel_source_sha256") != sha or rec.get("workload") != w.name:
        return None
    if launch is not None and rec.get("launch") != launch:
        return None
    try:
        return int(float(rec["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def cpu_baseline(w, inp, target_s: float = 12.0, max_rows: int | None = None, threads: int = 0):
    """Time the fp64 oracle (as it stands) on the host cores (all of them, or
    `threads`) over a sample of rows."""
    import oracle
    cores = threads if threads > 0 else len(os.sched_getaffinity(0))
    R = w.B * w.D
    rows = 64

    def run(nrows):
        # rows 0..nrows-1 of the flattened (B*D) rows: a contiguous prefix
        b_hi = (nrows + w.D - 1) // w.D
        x = inp["x"][:b_hi].reshape(-1, w.L)[:nrows]
        dl = inp["delta"][:b_hi].reshape(-1, w.L)[:nrows]
        # present the sample as (1, nrows, L) rows of batch 0 when it lies in batch 0
        if nrows <= w.D:
            args = (x[None], dl[None], inp["A"][:nrows], inp["Bm"][:1], inp["Cm"][:1],
                    inp["Dskip"][:nrows])
            t = time.perf_counter()
            oracle.selective_scan(*args, threads=cores)
            return time.perf_counter() - t
        ridx = np.arange(nrows)
        t = time.perf_counter()
        oracle.selective_scan(inp["x"], inp["delta"], inp["A"], inp["Bm"], inp["Cm"],
                              inp["Dskip"], rows=ridx, threads=cores)
        return time.perf_counter() - t

    rows = min(rows, R)
    dt = run(rows)
    while dt < target_s / 4 and rows < R and (max_rows is None or rows < max_rows):
        rows = min(R, rows * 4, max_rows or R)
        dt = run(rows)
    reps = 1
    import oracle as _o
    used = _o.threads_used(cores, rows)
    # the whole workload is short: repeat it until the sample is about 12 s of
    # CPU work (wall time x threads)
    while dt * used < 12.0 and dt < 30.0:
        reps *= 2
        dt = sum(run(rows) for _ in range(reps))
    elems = rows * w.L * w.N * reps
    return {
        "value": elems / dt, "unit": "elems/s", "cores": used,
        "kind": "oracle",
        "sample": f"{rows} of {R} (b,d) rows x L={w.L} x N={w.N} of {w.name}"
                  + (f", {reps} repeats" if reps > 1 else "") + f", fp64, {dt:.1f} s wall",
    }


def cpu_baseline_affine(w, inp, int32: bool, target_s: float = 8.0, threads: int = 0):
    """Time the bare-scan oracle (fp64, or the uint32 loop) over a sample of rows."""
    import oracle
    cores = threads if threads > 0 else len(os.sched_getaffinity(0))
    R = w.B * w.D
    a2, b2 = inp["a"].reshape(R, w.L), inp["bx"].reshape(R, w.L)
    rows, reps = min(R, 8), 1

    def run(nrows, nrep):
        t = time.perf_counter()
        for _ in range(nrep):
            if int32:
                oracle.affine_scan_i32(a2[:nrows], b2[:nrows], threads=cores)
            else:
                oracle.affine_scan(a2[:nrows], b2[:nrows], threads=cores)
        return time.perf_counter() - t

    dt = run(rows, reps)
    while dt < target_s / 4:
        if rows < R:
            rows = min(R, rows * 4)
        else:
            reps *= 4  # the whole workload is short: repeat it
        dt = run(rows, reps)
    return {
        "value": rows * w.L * reps / dt, "unit": "elems/s",
        "cores": oracle.threads_used(cores, rows), "kind": "oracle",
        "sample": f"{rows} of {R} rows x L={w.L} of {w.name}"
                  + (f", {reps} repeats" if reps > 1 else "")
                  + f", {'uint32' if int32 else 'fp64'}, {dt:.2f} s wall",
    }


def measure_copy_bandwidth(mib: int = 2048, reps: int = 10) -> dict:
    """A plain device-to-device copy of `mib` MiB, timed with HIP events:
    bytes read plus bytes written per second."""
    import torch
    n = mib << 18
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    sec = e0.elapsed_time(e1) * 1e-3 / reps
    return {"copy_GBs": 2 * n * 4 / sec / 1e9, "copy_MiB": mib, "reps": reps,
            "frac_of_peak": 2 * n * 4 / sec / 1e9 / HBM_PEAK_GBS}


SPREAD_LAUNCHES = 100


def clock_warmup(step, ms: float) -> int:
    """Launch steps until at least `ms` of wall time has passed (synchronising
    every few launches): the GPU raises its clock only after some tens of
    milliseconds of sustained work, and the first launches of a cold GPU run
    up to ~30% slower.  Returns the number of launches."""
    import torch
    if ms <= 0:
        return 0
    t0 = time.perf_counter()
    n = 0
    while (time.perf_counter() - t0) * 1e3 < ms:
        for _ in range(4):
            step(n)
            n += 1
        torch.cuda.synchronize()
    return n


def time_launches(step, steps, warmup):
    """Run `warmup` untimed steps, then exactly `steps` timed ones, back to back,
    between one pair of HIP events on the launch stream.

    Returns (wall seconds of the timed steps, GPU seconds per launch over them,
    per-launch seconds of a further untimed pass with an event pair around each
    launch).  The per-launch average comes from the timed region itself: event
    pairs around every launch put a marker between kernels that idles the GPU
    for a few microseconds each, so they are kept out of the timed region and
    serve only the spread (std, median) of the launch durations.
    """
    import torch
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for i in range(steps):
        step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_per = e0.elapsed_time(e1) * 1e-3 / max(steps, 1)
    n = min(steps, SPREAD_LAUNCHES)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(n)]
    for i in range(n):
        ev[i][0].record(stream)
        step(steps + i)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    spread = np.array([a.elapsed_time(b) * 1e-3 for a, b in ev])
    return wall, gpu_per, spread


GRAPH_SPREAD_REPLAYS = 20


def time_graph(step, steps, warmup):
    """time_launches with the launches replayed from a HIP graph.

    After `warmup` eager steps, `steps` launches are captured into one graph
    (torch's capture; the library enqueues on the capturing stream), which is
    replayed once untimed, then once between one pair of HIP events (exactly
    `steps` timed launches, without the host's per-call enqueue cost), then
    GRAPH_SPREAD_REPLAYS more times with an event pair around each replay for
    the spread (per-launch means of the replays).  Only calls that launch
    kernels and use no scratch or workspace can be captured; the library
    refuses the others while capturing.
    """
    import torch
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(3):
            step(i)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(steps):
            step(i)
    g.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_per = e0.elapsed_time(e1) * 1e-3 / max(steps, 1)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(GRAPH_SPREAD_REPLAYS)]
    for a, b in ev:
        a.record(stream)
        g.replay()
        b.record(stream)
    torch.cuda.synchronize()
    spread = np.array([a.elapsed_time(b) * 1e-3 / max(steps, 1) for a, b in ev])
    return wall, gpu_per, spread


def run_timed(step, args):
    args.clock_warmup_launches = clock_warmup(step, getattr(args, "clock_warmup_ms", 0))
    if getattr(args, "graph", False):
        return time_graph(step, args.steps, args.warmup)
    return time_launches(step, args.steps, args.warmup)


def warmup_record(args) -> dict:
    """How the GPU was warmed up before the timed steps (part of every line)."""
    return {"clock_warmup_ms": getattr(args, "clock_warmup_ms", 0),
            "clock_warmup_launches": getattr(args, "clock_warmup_launches", 0),
            "warmup_steps": args.warmup}


def launch_stats(gpu_per, spread, graph=False):
    """The per_launch_us object of a bench line."""
    out = {"mean": gpu_per * 1e6, "std": float(spread.std()) * 1e6,
           "median": float(np.median(spread)) * 1e6,
           "mean_of_spread_pass": float(spread.mean()) * 1e6, "spread_launches": len(spread),
           "method": "mean: HIP events around the timed steps / steps; std, median: an "
                     "untimed pass after them with an event pair around each launch"}
    if graph:
        del out["spread_launches"]  # the spread is over replays, not single launches
        out["spread_replays"] = len(spread)
        out["method"] = ("launches replayed from one HIP graph of `steps` launches; mean: HIP "
                         "events around one replay / steps; std, median: over the per-launch "
                         "means of further replays, an event pair around each")
    return out


def bench_affine(w, args):
    """The bare affine scan (fp32): an HBM-bound kernel, 12 bytes per element."""
    import torch

    import paper_2606_00601_amd as sw
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sw.lib()
    inp = w.inputs()
    if args.int32:
        inp = wl.affine_inputs_i32(w.B, w.D, w.L, wl.INT_SEEDS["uniform"], "uniform")
    proj = args.form == "proj"
    # bare: a, bx read, h written; projection form (Eq. (3)-(4)): a, b, x, c
    # read, y written, h_last written once per row
    abytes = (20 if proj else 12) * w.elems + (4 * w.B * w.D if proj else 0)
    nsets = args.sets or max(1, min(4, int(np.ceil(2 * MALL_BYTES / abytes)) + 1))
    if proj:
        rng = np.random.Generator(np.random.PCG64(w.seed + 100))
        xc = [rng.standard_normal(size=(w.B, w.D, w.L)).astype(np.float32) for _ in range(2)]
    sets = []
    for i in range(nsets):
        a = torch.from_numpy(inp["a"]).to(dev)
        bx = torch.from_numpy(inp["bx"]).to(dev)
        extra = tuple(torch.from_numpy(v).to(dev) for v in xc) if proj else ()
        sets.append((a, bx, torch.empty_like(a)) + extra)
    cpu = None if args.no_cpu or proj else cpu_baseline_affine(w, inp, args.int32,
                                                               threads=args.cpu_threads)
    del inp

    def step(i):
        st = sets[i % nsets]
        a, bx, h = st[:3]
        if proj:
            sw.affine_scan_proj(a, bx, st[3], st[4], y=h)
        elif args.int32:
            sw.affine_scan_i32(a, bx, out=h)
        elif args.schedule == "default":
            sw.affine_scan(a, bx, out=h)
        else:
            sw.affine_scan_schedule(a, bx, out=h, schedule=args.schedule)

    wall, kern, per = run_timed(step, args)
    gbs = abytes / kern / 1e9
    # the library walks each row in one workgroup once the rows alone fill the
    # GPU (>= 8 per CU) and a row is longer than one 2048-step chunk
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    kname = ("affine_rows_kernel" if w.L > 2048 and w.B * w.D >= 8 * cus
             else "affine_scan_kernel")
    if args.schedule == "blelloch":
        kname = "affine_blelloch_kernel"
    if proj:
        kname += " (projection variant)"
    out = {
        "metric": ("affine-scan fwd, projection form y = c*h, h = a*h + b*x, B*L*D elems/s "
                   "(+ achieved HBM GB/s vs peak), 1 GPU" if proj else
                   "affine-scan fwd B*L*D elems/s (+ achieved HBM GB/s vs peak), 1 GPU"),
        "value": w.elems * args.steps / wall, "unit": "elems/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int32" if args.int32 else "f32", "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "D": w.D, "L": w.L, "input_sets_rotated": nsets,
                   "schedule": args.schedule, "form": args.form,
                   "launch": "hip-graph" if args.graph else "eager",
                   "warmup": warmup_record(args)},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS,
                     "traffic": (measured_traffic(w) if args.schedule == "default" and not proj
                                 and not args.int32 else None),
                     "kernel": kname,
                     "per_launch_us": launch_stats(kern, per, args.graph)},
    }
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)
    return 0


# fp32 flops the backward needs per (b,d,t,n) element (the exp2 not counted):
# twelve operations -- delta*A', (delta*x)*B, a*h_{t-1}, the state add, the
# adjoint FMA, lam*q, the dA FMA, (lam q)*A, lam*B, lam*(delta x), ds*h and
# a*lam -- two of them FMAs (the forward sweep that rebuilds the tile
# checkpoints is overhead)


def bench_bwd(w, args):
    """Backward of the fused scan on the same workload: dy in the input dtype,
    every gradient in fp32."""
    import torch

    import paper_2606_00601_amd as sw
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sw.lib()
    inp = w.inputs()
    rng = np.random.Generator(np.random.PCG64(4242))
    dy = rng.standard_normal((w.B, w.D, w.L)).astype(np.float32)
    es = 2 if w.dtype == "bf16" else 4
    if w.dtype == "bf16":
        dy_t = torch.from_numpy(wl.bf16_round(dy).view(np.int16)).to(dev).view(torch.bfloat16)
    else:
        dy_t = torch.from_numpy(dy).to(dev)

    def to_dev(k):
        if w.dtype == "bf16" and k in ("x", "delta", "Bm", "Cm"):
            return torch.from_numpy(inp[k + "_bf16"].view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(inp[k]).to(dev)

    t = {k: to_dev(k) for k in ("x", "delta", "A", "Bm", "Cm", "Dskip")}
    del inp
    opt = {}
    if args.options:
        # the Mamba-block inputs: gate z (the input dtype), delta bias with
        # softplus, initial state
        orng = np.random.Generator(np.random.PCG64(w.seed + 200))
        z = orng.standard_normal(size=(w.B, w.D, w.L)).astype(np.float32)
        opt["z"] = (torch.from_numpy(wl.bf16_round(z).view(np.int16)).to(dev).view(torch.bfloat16)
                    if w.dtype == "bf16" else torch.from_numpy(z).to(dev))
        opt["delta_bias"] = torch.from_numpy(
            orng.uniform(-2.0, 0.0, size=w.D).astype(np.float32)).to(dev)
        opt["h0"] = torch.from_numpy(
            orng.standard_normal(size=(w.B, w.D, w.N)).astype(np.float32)).to(dev)
        opt["delta_softplus"] = True

    ck = sp = None
    if args.ckpt:
        # the forward's checkpoints (and, with the gate, its output before the
        # gate), as a training step would hand them over
        ck = sw.new_ckpt(t["x"], w.N)
        if "z" in opt:
            sp = torch.empty((w.B, w.D, w.L), dtype=torch.float32, device=dev)
        sw.selective_scan_fwd(t["x"], t["delta"], t["A"], t["Bm"], t["Cm"], t["Dskip"], ckpt=ck,
                              s_pre=sp, **opt)
        torch.cuda.synchronize()

    def step(i):
        sw.selective_scan_bwd(t["x"], t["delta"], t["A"], t["Bm"], t["Cm"], t["Dskip"], dy_t,
                              ckpt=ck, s_pre=sp, **opt)

    wall, kern, per = run_timed(step, args)
    launch = sw.last_launch()  # the backward's kernels and where its checkpoints came from
    elems = w.elems
    # algorithmic bytes: x, delta, dy read; dx, ddelta written (fp32); B, C
    # read, dB, dC written (fp32); A, Dskip read, dA, dDskip, dh0 written
    abytes = (3 * es + 8) * w.B * w.D * w.L + (2 * es + 8) * w.B * w.L * w.N \
        + 8 * w.D * w.N + 8 * w.D + 4 * w.B * w.D * w.N
    if args.options:
        # z read, dz written; delta bias read, its gradient written; h0 read
        abytes += (es + 4) * w.B * w.D * w.L + 8 * w.D + 4 * w.B * w.D * w.N
    flops = FLOP_PER_ELEM_BWD * elems / kern
    gbs = abytes / kern / 1e9
    out = {
        "metric": "selective-scan bwd B*L*D*N elems/s (all gradients), 1 GPU",
        "value": elems * args.steps / wall, "unit": "elems/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "D": w.D, "N": w.N, "L": w.L,
                   "pass": "backward", "dy": w.dtype, "gradients": "fp32",
                   "options": ("gate z, delta bias + softplus, initial state" if args.options
                               else "none"),
                   "forward_checkpoints": bool(args.ckpt), "warmup": warmup_record(args)},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS,
                     "traffic": (measured_traffic(w, bwd=True)
                                 if args.ckpt and not args.options else None),
                     "kernel": launch,
                     "per_launch_us": launch_stats(kern, per, args.graph),
                     "algorithmic_bytes": abytes},
        "alu": {"achieved": flops / 1e12, "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": flops / 1e12 / FP32_PEAK_TFLOPS, "flop_per_elem": FLOP_PER_ELEM_BWD},
    }
    print(json.dumps(out), flush=True)
    return 0


# shapes of --layout-sweep: D from 1/3 to 2 wavefronts per SIMD at one lane per
# state and B = 1, three lengths, and a few with B > 1
LAYOUT_SWEEP_SHAPES = ";".join(
    [f"1,{D},{L}" for L in (4096, 16384, 65536) for D in (1280, 2560, 4096, 5120, 6144, 8192)]
    + ["2,2560,8192", "4,1024,16384", "2,2048,32768"])

# forced choices of the N = 16 forward (environment of the library) timed by --layout-sweep
LAYOUT_CANDIDATES = (
    [("whole", {"SW_SS_QUAD": "0", "SW_SS_SEGMENTS": "1"})]
    + [(f"r16c{k}", {"SW_SS_QUAD": "0", "SW_SS_SEGMENTS": str(k), "SW_SS_SEGFORM": "2"})
       for k in (2, 4, 6, 8, 16)]
    + [(f"r16r{k}", {"SW_SS_QUAD": "0", "SW_SS_SEGMENTS": str(k), "SW_SS_SEGFORM": "1"})
       for k in (4, 8)]
    + [(f"quad{k}", {"SW_SS_QUAD": "1", "SW_SS_SEGMENTS": str(k)}) for k in (4, 8, 9, 12, 16)])


def layout_sweep(shapes: str) -> int:
    """Time each forced layout / segment count / form of the fused forward and
    the library's own choice on seeded synthetic inputs (Mamba-like: delta =
    softplus(N(-4, 0.5^2)), A = -exp(U[0, ln 16]), x, B, C, Dskip standard
    normal), fp32 and bf16 inputs, N = 16; one JSON line per shape."""
    import torch

    import paper_2606_00601_amd as sw
    sw.lib()
    dev = torch.device("cuda:0")
    keys = ("SW_SS_QUAD", "SW_SS_SEGMENTS", "SW_SS_SEGFORM")
    saved = {k: os.environ.get(k) for k in keys}
    g = torch.Generator(device=dev)
    g.manual_seed(1)
    clock_warmup(lambda i: torch.cumsum(torch.ones(1 << 24, device=dev), 0), 250.0)
    for dt in ("f32", "bf16"):
        for spec in shapes.split(";"):
            B, D, L = (int(v) for v in spec.split(","))
            N = 16
            x = torch.randn(B, D, L, device=dev, generator=g)
            dl = torch.nn.functional.softplus(
                torch.randn(B, D, L, device=dev, generator=g) * 0.5 - 4)
            A = -torch.exp(torch.rand(D, N, device=dev, generator=g) * float(np.log(16)))
            Bm = torch.randn(B, L, N, device=dev, generator=g)
            Cm = torch.randn(B, L, N, device=dev, generator=g)
            if dt == "bf16":
                x, dl, Bm, Cm = x.bfloat16(), dl.bfloat16(), Bm.bfloat16(), Cm.bfloat16()
            Dk = torch.randn(D, device=dev, generator=g)
            y = torch.empty(B, D, L, device=dev)
            h = torch.empty(B, D, N, device=dev)

            def call():
                sw.selective_scan_fwd(x, dl, A, Bm, Cm, Dk, y=y, h_last=h)

            n = max(10, min(60, int(4e9 / (B * D * L))))
            res = {}
            for name, env in LAYOUT_CANDIDATES + [("auto", {})]:
                for k in keys:
                    os.environ.pop(k, None)
                os.environ.update(env)
                for _ in range(max(3, n // 4)):
                    call()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                torch.cuda.synchronize()
                e0.record()
                for _ in range(n):
                    call()
                e1.record()
                torch.cuda.synchronize()
                res[name] = round(1e3 * e0.elapsed_time(e1) / n, 1)
                if name == "auto":
                    res["auto_launch"] = sw.last_launch()
            for k in keys:
                os.environ.pop(k, None)
            best = min((v, k) for k, v in res.items() if k not in ("auto", "auto_launch"))
            print(json.dumps({"B": B, "D": D, "L": L, "N": N, "inputs": dt, "us": res,
                              "fastest_forced": best[1],
                              "auto_over_fastest": round(res["auto"] / best[0], 3)}),
                  flush=True)
    for k, v in saved.items():
        if v is not None:
            os.environ[k] = v
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    # the GPU reaches its steady clock only after some tens of milliseconds of
    # sustained launches (the first ~30 ms run up to ~30% slower): launches run
    # for at least this long before the W warm-up steps, whatever W is
    ap.add_argument("--clock-warmup-ms", type=float, default=250.0)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(wl.WORKLOADS))
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="host threads for the CPU oracle baseline (0: all cores)")
    ap.add_argument("--int32", action="store_true",
                    help="bare-scan workloads: the int32 wraparound mode")
    ap.add_argument("--measure-copy", action="store_true",
                    help="only time a plain 2 GiB device copy and print its bandwidth")
    ap.add_argument("--pass", dest="which", choices=("fwd", "bwd"), default="fwd",
                    help="time the forward (default, the headline metric) or the backward")
    ap.add_argument("--schedule", choices=("default", "blelloch"), default="default",
                    help="scan schedule of the bare-scan workloads (schedule ablation)")
    ap.add_argument("--ckpt", action="store_true",
                    help="training mode: the forward writes 8-step checkpoints, the backward "
                         "takes them")
    ap.add_argument("--options", action="store_true",
                    help="with the Mamba-block inputs (gate, delta bias + softplus, initial "
                         "state; the forward's y in the input dtype), forward or backward")
    ap.add_argument("--form", choices=("bare", "proj"), default="bare",
                    help="bare-scan workloads: the plain scan or the Eq. (3)-(4) projection form")
    ap.add_argument("--sets", type=int, default=0,
                    help="input sets rotated through (default: enough to exceed the MALL)")
    ap.add_argument("--print-kernel-sha", action="store_true",
                    help="print the hash of the kernel sources of --workload's path "
                         "(the key of its traffic record) and exit")
    ap.add_argument("--graph", action="store_true",
                    help="replay the timed launches from one HIP graph (forward and bare "
                         "scan; removes the host's per-call enqueue cost, which bounds the "
                         "launch-sized workloads)")
    ap.add_argument("--layout-sweep", action="store_true",
                    help="time every layout, segment count and form of the N = 16 fused "
                         "forward, and the library's own choice, over --sweep-shapes "
                         "(one JSON line per shape and input dtype)")
    ap.add_argument("--sweep-shapes", default=LAYOUT_SWEEP_SHAPES,
                    help="B,D,L triples separated by ';' for --layout-sweep")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB, 5 times "
                         "(reference kernel for scaling the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(rows shard across GPUs without communication; see the design notes).",
              file=sys.stderr)
        return 2

    if args.print_kernel_sha:
        print(kernel_source_sha256("bwd" if args.which == "bwd" else wl.workload(args.workload).path))
        return 0

    import torch

    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib << 18  # fp32 elements
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "copy", "bytes_read": n * 4, "bytes_written": n * 4,
                          "launches": 5}), flush=True)
        return 0

    if args.measure_copy:
        print(json.dumps(measure_copy_bandwidth()), flush=True)
        return 0

    if args.layout_sweep:
        return layout_sweep(args.sweep_shapes)

    import paper_2606_00601_amd as sw
    w = wl.workload(args.workload)
    if args.graph and args.which == "bwd":
        print("--graph: the backward allocates a workspace per call and cannot be captured",
              file=sys.stderr)
        return 2
    if w.path == "affine":
        return bench_affine(w, args)
    if args.which == "bwd":
        return bench_bwd(w, args)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sw.lib()  # the HIP library must be present: no fallback

    inp = w.inputs()
    abytes = algorithmic_bytes(w)
    es = 2 if w.dtype == "bf16" else 4
    if args.options:
        # + z read, h0 read, delta_bias read; y written in the input dtype
        abytes += es * w.B * w.D * w.L + 4 * w.B * w.D * w.N + 4 * w.D
        abytes -= (4 - es) * w.B * w.D * w.L
    if args.ckpt:
        abytes += 4 * w.B * w.D * ((w.L + 7) // 8) * 16  # the checkpoints written
    nsets = args.sets or max(2, int(np.ceil(2 * MALL_BYTES / abytes)) + 1)
    nsets = min(nsets, 8)

    def to_dev(k):
        if w.dtype == "bf16" and k in ("x", "delta", "Bm", "Cm"):
            return torch.from_numpy(inp[k + "_bf16"].view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(inp[k]).to(dev)

    base = {k: to_dev(k) for k in ("x", "delta", "A", "Bm", "Cm", "Dskip")}
    opt = {}
    y_dtype = torch.float32
    if args.options:
        # the Mamba-block inputs: gate z, delta bias with softplus, initial state,
        # y in the input dtype
        rng = np.random.Generator(np.random.PCG64(w.seed + 200))
        z = rng.standard_normal(size=(w.B, w.D, w.L)).astype(np.float32)
        if w.dtype == "bf16":
            opt["z"] = torch.from_numpy(wl.bf16_round(z).view(np.int16)).to(dev).view(
                torch.bfloat16)
            y_dtype = torch.bfloat16
        else:
            opt["z"] = torch.from_numpy(z).to(dev)
        opt["delta_bias"] = torch.from_numpy(
            rng.uniform(-2.0, 0.0, size=w.D).astype(np.float32)).to(dev)
        opt["h0"] = torch.from_numpy(
            rng.standard_normal(size=(w.B, w.D, w.N)).astype(np.float32)).to(dev)
        opt["delta_softplus"] = True
    sets = []
    for i in range(nsets):
        s = {k: (v if i == 0 else v.clone()) for k, v in base.items()}
        s["y"] = torch.empty((w.B, w.D, w.L), dtype=y_dtype, device=dev)
        s["h"] = torch.empty((w.B, w.D, w.N), dtype=torch.float32, device=dev)
        if args.ckpt:
            s["ck"] = sw.new_ckpt(s["x"], w.N)
        sets.append(s)
    torch.cuda.synchronize()

    def step(i):
        s = sets[i % nsets]
        if args.schedule == "default":
            sw.selective_scan_fwd(s["x"], s["delta"], s["A"], s["Bm"], s["Cm"], s["Dskip"],
                                  y=s["y"], h_last=s["h"], y_dtype=y_dtype, ckpt=s.get("ck"),
                                  **opt)
        else:
            sw.selective_scan_fwd_schedule(s["x"], s["delta"], s["A"], s["Bm"], s["Cm"],
                                           s["Dskip"], schedule=args.schedule)

    step(0)
    launch = sw.last_launch()  # the kernels the library picked for this call
    wall, kern, per = run_timed(step, args)

    elems = w.elems
    value = elems * args.steps / wall
    hbm_gbs = abytes / kern / 1e9
    flops = FLOP_PER_ELEM * elems / kern
    fwd_kernel = launch
    out = {
        "metric": "selective-scan fwd B*L*D*N elems/s (+ achieved HBM GB/s vs peak), 1 GPU",
        "value": value,
        "unit": "elems/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": w.name, "B": w.B, "D": w.D, "N": w.N, "L": w.L,
            "inputs": ("bf16 x/delta/Bm/Cm, fp32 A/Dskip" if w.dtype == "bf16" else "fp32"),
            "state_and_output": "fp32" if y_dtype == torch.float32 else "fp32 state, bf16 y",
            "input_sets_rotated": nsets, "schedule": args.schedule,
            "options": ("gate z, delta bias + softplus, initial state" if args.options
                        else "none"),
            "forward_checkpoints": bool(args.ckpt),
            "launch": "hip-graph" if args.graph else "eager",
            "warmup": warmup_record(args),
        },
        "roofline": {
            "bound": "hbm",
            "achieved": hbm_gbs,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": hbm_gbs / HBM_PEAK_GBS,
            "traffic": (measured_traffic(w, launch) if args.schedule == "default"
                        and not args.options and not args.ckpt else None),
            "kernel": fwd_kernel,
            "per_launch_us": launch_stats(kern, per, args.graph),
            "algorithmic_bytes": abytes,
        },
        "alu": {"achieved": flops / 1e12, "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": flops / 1e12 / FP32_PEAK_TFLOPS, "flop_per_elem": FLOP_PER_ELEM},
    }
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(w, inp, threads=args.cpu_threads)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
