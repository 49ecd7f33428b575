#!/usr/bin/env python3
"""Benchmark: Sparse DNN Challenge inference (Kepner et al., 2019) on one MI355X.

A step is the challenge's timed region (Sec. V): evaluate every layer for all input rows and identify
the categories -- one sdnn_infer + sdnn_categories through the C ABI, with the inputs and weights
already resident in HBM. The metric is the paper's rate (Sec. V, Sec. VI-B):
(# inputs) x (# connections) / time, in inputs*edges/s.

Workloads are the seeded synthetic stand-ins for the paper's networks and MNIST-derived inputs
(synth.CONFIGS; Table 1 widths and biases, Table 2 depths). The default is the 65536-neuron,
1920-layer network on 60,000 inputs, on the library's default kernels, which read every edge's
weight and every neuron's bias from memory. --equal-value-kernels measures the opt-in kernels that
exploit the workloads' equal weights and biases instead (a supplementary line: the paper's Sec. V
lists exploiting repeated weight and bias values among what a submission should avoid).

Prints ONE JSON line on stdout; progress goes to stderr.
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

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published


def log(msg: str) -> None:
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def algorithmic_layer_bytes(n: int, nnz: int, r_in: int, r_out: int) -> int:
    """Bytes one layer must move with dense fp32 live rows: read the live input rows, write the rows
    that stay live, read the weights (index + value) and the bias once. Every column counts, also
    where columns are equal (the method computes each of them)."""
    if r_in == 0:
        return 0
    return 4 * n * (r_in + r_out) + 8 * nnz + 4 * n


def layer_source(cfg, network: str):
    """The weight layers of a workload: the configs' permutation-union layers, or structured
    RadiX-Net style layers of the same width (synth.radix_layers_csc)."""
    import synth
    if network == "radix":
        return lambda l0, nl: synth.radix_layers_csc(cfg.net_id, l0, nl, cfg.n_neurons, cfg.weight)
    return lambda l0, nl: synth.layers_csc(cfg.net_id, l0, nl, cfg.n_neurons, cfg.k, cfg.weight)


def workload_name(cfg, network: str, equal_values: bool = False) -> str:
    name = cfg.name if network == "union" else f"{network}-{cfg.name}"
    return name + ("-eqv" if equal_values else "")


def host_cpus() -> dict:
    """The host's CPUs as this process sees them: os.cpu_count() (nproc of the machine), the CPUs in
    this process's affinity mask, the cgroup CPU quota (cpu.max, if any), the usable count (the
    smallest of those), and the CPU model string."""
    nproc = os.cpu_count() or 1
    try:
        affinity = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        affinity = nproc
    quota = None
    try:
        with open("/sys/fs/cgroup/cpu.max") as f:
            q, period = f.read().split()[:2]
        if q != "max":
            quota = max(1, int(int(q) // int(period)))
    except (OSError, ValueError):
        quota = None
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    usable = min(x for x in (nproc, affinity, quota) if x)
    return {"nproc": nproc, "affinity": affinity, "cgroup_quota": quota, "usable": usable, "model": model}


# The supplementary all-live input set: Bernoulli(0.6) rows. Each column sums 32 weights of 1/16,
# so a row grows while its mean exceeds -b; at density 0.6 every row stays live at every width and
# saturates at YMAX within a few layers, so each layer runs at its full shape (R_l = M).
ALL_LIVE_DENSITY = 0.6


def workload(cfg, inputs: str, layers: int | None):
    """The config, cut to its first `layers` layers and, for the all-live set, renamed."""
    import dataclasses
    L = layers or cfg.n_layers
    if L == cfg.n_layers and inputs == "strokes":
        return cfg
    name = f"n{cfg.n_neurons}-l{L}-m{cfg.n_rows}"
    return dataclasses.replace(cfg, n_layers=L, name=("alllive-" + name) if inputs == "alllive" else name)


def input_rows(cfg, inputs: str, r0: int, nr: int) -> np.ndarray:
    """Rows [r0, r0 + nr) of the workload's inputs: the config's stroke images, or Bernoulli rows."""
    import synth
    if inputs == "alllive":
        return synth.inputs(cfg.input_set, cfg.side, r0, nr, "bernoulli", ALL_LIVE_DENSITY)
    return synth.config_inputs(cfg, r0, nr)


def cpu_baseline(cfg, target_s: float, threads: int, network: str = "union", inputs: str = "strokes") -> dict:
    """The oracle as it is, on a bounded sample of the same workload (first rows of the input set),
    timing only its layer evaluations (weight generation is loading, untimed as on the GPU side)."""
    import oracle
    layers = layer_source(cfg, network)

    def run(rows: int) -> float:
        y0 = input_rows(cfg, inputs, 0, rows)
        o = oracle.Oracle(y0, cfg.ymax)
        bias = np.full(cfg.n_neurons, cfg.bias, np.float32)
        spent, l, chunk = 0.0, 0, 8
        while l < cfg.n_layers and o.live > 0:
            nl = min(chunk, cfg.n_layers - l)
            cp, ri, v = layers(l, nl)
            for i in range(nl):
                t0 = time.perf_counter()
                o.layer(cp[i], ri, v, bias, threads)
                spent += time.perf_counter() - t0
                if o.live == 0:
                    break
            l += nl
        cats = o.categories().size
        o.close()
        log(f"cpu baseline: {rows} rows in {spent:.2f} s ({cats} categories)")
        return spent

    rows = min(cfg.n_rows, 64)
    t = run(rows)
    while t < target_s / 3 and rows < cfg.n_rows:
        rows = int(min(cfg.n_rows, max(rows * 2, rows * target_s / max(t, 1e-3))))
        t = run(rows)
    rate = rows * cfg.total_nnz / t
    cpus = host_cpus()
    return {"value": rate, "unit": "inputs*edges/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpus["model"], "nproc": cpus["nproc"], "affinity_cpus": cpus["affinity"],
            "cgroup_cpu_quota": cpus["cgroup_quota"],
            "sample": f"first {rows} of {cfg.n_rows} input rows of {workload_name(cfg, network)}, all {cfg.n_layers} layers "
                      f"(rows stop when dead, as on the GPU); {t:.2f} s of oracle layer evaluation on "
                      f"{threads} host threads (every CPU this process may use: the smallest of nproc "
                      f"{cpus['nproc']}, its affinity mask {cpus['affinity']} and the cgroup quota "
                      f"{cpus['cgroup_quota']}); {cpus['model']}"}


def calibrate_copy(nbytes: int) -> int:
    """A plain device-to-device copy of known size, run under rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE
    to scale those counters to bytes."""
    import torch
    a = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes": nbytes}))
    return 0


def copy_bandwidth(nbytes: int = 1 << 30, reps: int = 5) -> float:
    """Measured device-to-device copy rate in GB/s (bytes read + bytes written over the time, HIP
    events on the current stream, best of `reps`): the practical HBM ceiling beside the published
    peak."""
    import torch
    a = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    best = float("inf")
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        b.copy_(a)
        e1.record()
        e1.synchronize()
        best = min(best, e0.elapsed_time(e1) * 1e-3)
    del a, b
    return 2 * nbytes / best / 1e9


def source_code_sha(text: str) -> str:
    """SHA-256 of C/HIP source text with comments removed and whitespace collapsed: it changes with
    the code and not with its comments."""
    import hashlib
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return hashlib.sha256(" ".join(text.split()).encode()).hexdigest()


def kernel_source_sha() -> str:
    with open(os.path.join(ROOT, "paper_1909_05631_amd", "csrc", "sdnn.hip")) as f:
        return source_code_sha(f.read())


def committed_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` measured with rocprofv3 counters for this workload, if the
    record in profiles/ was taken with the current kernel source; None otherwise."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != kernel_source_sha() or rec.get("kernel") != kernel:
        return None
    return rec.get("bytes_per_launch")


def committed_lds(workload: str, kernel: str):
    """LDS bank-conflict share (bank-conflict stall cycles over LDS-active cycles, rocprofv3
    SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE) of each kernel of `kernel` (names joined by '+'), from
    the same record as committed_traffic; None if absent or taken with another kernel source."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_sha256") != kernel_source_sha() or "lds" not in rec:
        return None
    parts = kernel.split("+")
    out = {k: v["conflict_cycle_frac"] for k, v in rec["lds"]["kernels"].items() if k.split("<")[0] in parts}
    return out or None


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=4, help="index into synth.CONFIGS (0-4)")
    ap.add_argument("--network", choices=["union", "radix"], default="union",
                    help="weight layers: the configs' permutation unions, or structured RadiX-Net style "
                         "layers (Kronecker-expanded radix-2 base DNN, Fig. 1 / Table 1) of the same width")
    ap.add_argument("--inputs", choices=["strokes", "alllive"], default="strokes",
                    help="the config's stroke images (~19%% ones), or the supplementary all-live set "
                         "(Bernoulli(0.6) rows: every row stays live, so every layer runs at full shape)")
    ap.add_argument("--layers", type=int, default=0, help="run only the first LAYERS layers (0: all)")
    ap.add_argument("--shard", type=int, default=1, metavar="G",
                    help="time one GPU's share of a G-GPU data-parallel split (rows are interleaved: this is "
                         "the share of GPU 0, input rows i with i %% G == 0); no CPU baseline")
    ap.add_argument("--equal-value-kernels", action="store_true",
                    help="supplementary: opt in to the kernels that exploit layers whose weights and biases "
                         "are all equal (sdnn_enable_equal_value_kernels); the workload name gets '-eqv'")
    ap.add_argument("--profile-steps", type=int, default=2,
                    help="untimed steps run after the timed ones with per-layer events, for the roofline")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU-baseline time")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip the per-layer events (no roofline)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only copy BYTES between two device buffers (for scaling HBM byte counters)")
    args = ap.parse_args()
    if args.calibrate_copy:
        return calibrate_copy(args.calibrate_copy)

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: it measures the single-GPU share of the "
              "data-parallel path (inputs split across GPUs, weights replicated); use --gpus 1.",
              file=sys.stderr)
        return 2

    import torch

    import synth
    from paper_1909_05631_amd import sdnn

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    torch.cuda.set_device(0)
    cfg = workload(synth.CONFIGS[args.config], args.inputs, args.layers)
    if args.shard < 1:
        print("--shard needs G >= 1", file=sys.stderr)
        return 2
    G = args.shard
    n, L = cfg.n_neurons, cfg.n_layers
    m = (cfg.n_rows + G - 1) // G  # rows 0, G, 2G, ... of the workload
    wname = workload_name(cfg, args.network, args.equal_value_kernels) + (f"-shard0of{G}" if G > 1 else "")
    layers = layer_source(cfg, args.network)
    stream = torch.cuda.current_stream()

    # ---------------- untimed: load the network and inputs into HBM (Sec. V, load steps)
    t0 = time.time()
    y0 = torch.empty((m, n), dtype=torch.float32, device="cuda")
    chunk = max(G, (1 << 28) // (4 * n) // G * G)
    for r0 in range(0, cfg.n_rows, chunk):
        nr = min(chunk, cfg.n_rows - r0)
        rows = input_rows(cfg, args.inputs, r0, nr)[::G]  # r0 is a multiple of G
        y0[r0 // G:r0 // G + rows.shape[0]].copy_(torch.from_numpy(np.ascontiguousarray(rows)))
    density = float(y0.mean().item())
    log(f"{wname}: inputs on device ({m} x {n}, density {density:.3f}) in {time.time() - t0:.1f} s")
    t0 = time.time()
    net = sdnn.Net(n, L, cfg.ymax, equal_value_kernels=args.equal_value_kernels)
    lchunk = max(1, min(64, (1 << 27) // (n * cfg.k)))
    for l0 in range(0, L, lchunk):
        nl = min(lchunk, L - l0)
        cp, ri, v = layers(l0, nl)
        net.load_layers(l0, cp, ri, v, np.full((nl, n), cfg.bias, np.float32))
        if (l0 // lchunk) % 8 == 0:
            log(f"loaded layers {l0 + nl}/{L}")
    log(f"network loaded ({L} layers, {cfg.total_nnz} connections) in {time.time() - t0:.1f} s; "
        f"kernel path {net.kernel_path}")
    nb = net.workspace_bytes(m)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()

    def step():
        net.infer(y0, m, ws, nb, stream)
        return net.categories()

    for i in range(args.warmup):
        cats = step()
        log(f"warmup {i}: {cats.size} categories")
    # the timed steps run with per-layer events off; the events are taken in a separate pass below
    net.set_profiling(False)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        cats = step()
    torch.cuda.synchronize()
    t_total = time.perf_counter() - t_start
    t_step = t_total / max(args.steps, 1)
    counts = net.live_counts()
    log(f"timed {args.steps} steps: {t_step * 1e3:.3f} ms/step; categories {cats.size}; "
        f"live counts {counts[:8].tolist()}")

    edges = m * cfg.total_nnz
    value = edges / t_step
    nnz = cfg.nnz_per_layer
    live_edges = int(sum(int(counts[l]) * nnz for l in range(L)))

    roofline = None
    if not args.no_profile:
        # untimed pass with HIP events on the library's stream around the large layers only
        # (recording them around every layer of the long tail would slow what they measure)
        net.set_profiling(True, large_only=True)
        for _ in range(max(1, args.profile_steps)):
            step()
        net.set_profiling(False)
        # the dominant kernel: the large layer with the most event time; its launches are the rounds
        # (or the pack + layer pair) that the event pair of that layer spans
        ms, runs = net.layer_times()
        kind, launches = net.layer_info()
        per_run = ms / np.maximum(runs, 1)
        timed = [l for l in range(L) if runs[l] > 0]
        lay = max(timed, key=lambda l: per_run[l])
        # a launch that runs every remaining layer (kind 8) is timed at its first layer and covers
        # the algorithmic bytes of all of them
        covered = range(lay, L) if sdnn.KERNEL_KINDS.get(int(kind[lay])) == "k_layers_lds" else [lay]
        def layer_bytes(l):
            return algorithmic_layer_bytes(n, nnz, int(counts[l]), int(counts[l + 1]))

        algo = sum(layer_bytes(l) for l in covered)
        nl = max(int(launches[lay]), 1)
        avg_launch_ms = float(per_run[lay]) / nl
        achieved = algo / nl / (avg_launch_ms * 1e-3) / 1e9
        kname = sdnn.KERNEL_KINDS.get(int(kind[lay]), str(int(kind[lay])))
        head = ", ".join(f"{l}:{per_run[l] * 1e3:.1f}us({sdnn.KERNEL_KINDS.get(int(kind[l]))} x{int(launches[l])}, "
                         f"R={int(counts[l])})" for l in timed[:6])
        log(f"large-layer kernel times: {head}")
        def timed_bytes(l):
            cov = range(l, L) if sdnn.KERNEL_KINDS.get(int(kind[l])) == "k_layers_lds" else [l]
            return sum(layer_bytes(q) for q in cov)
        tot_bytes = sum(timed_bytes(l) * int(runs[l]) for l in timed)
        tot_ms = float(ms[timed].sum())
        copy_gbs = copy_bandwidth()
        roofline = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 5), "traffic": committed_traffic(wname, kname),
                    "lds_bank_conflict": committed_lds(wname, kname),
                    "copy_gbs": round(copy_gbs, 1), "frac_of_copy": round(achieved / copy_gbs, 5),
                    "kernel": kname, "layer": lay, "launches_per_step": nl,
                    "avg_launch_ms": round(avg_launch_ms, 5), "algorithmic_bytes_per_launch": int(algo / nl),
                    "large_layers": {"layers": len(timed),
                                     "achieved": round(tot_bytes / (tot_ms * 1e-3) / 1e9, 2) if tot_ms > 0 else None}}

    cpu = None
    if not args.no_cpu_baseline and G == 1:
        cpu = cpu_baseline(cfg, args.cpu_seconds, host_cpus()["usable"], args.network, args.inputs)

    out = {
        "metric": "inference edges/sec (Ninputs*sum nnz(W)/t) + % HBM roofline, 1 MI355X",
        "value": value,
        "unit": "inputs*edges/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t_step * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wname, "network": "permutation-union" if args.network == "union" else "radix-kronecker",
                   "kernels": ("supplementary: opt-in kernels exploiting equal weights and biases"
                               if args.equal_value_kernels else
                               "default: every edge's weight and every neuron's bias read from memory"),
                   "n_neurons": n, "n_layers": L, "n_rows": m, "bias": cfg.bias,
                   "ymax": cfg.ymax, "connections": cfg.total_nnz, "input_density": round(density, 4),
                   "inputs": "binary stroke images" if args.inputs == "strokes" else
                             f"binary Bernoulli({ALL_LIVE_DENSITY}) rows, all live (supplementary set)",
                   "parallelism": "none (1 GPU)" if G == 1 else
                                  f"GPU 0's share of a {G}-GPU row split (rows i % {G} == 0), timed on 1 GPU"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "live_edges_per_s": live_edges / t_step,
        "categories": int(cats.size),
        "live_counts_head": [int(c) for c in counts[:8]],
        # kernel family of each of the first 8 layers of the last run (sdnn_layer_info)
        "layer_kernels_head": [sdnn.KERNEL_KINDS.get(int(k), str(int(k))) for k in net.layer_info()[0][:8]],
    }
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
