#!/usr/bin/env python3
"""Benchmark of the temporally fused LIF layer on one MI355X.

Default step = the fused forward plus the fused backward of the conv-shaped LIF layer
x[T=16, B=64, C=128, H=32, W=32] (fp32 I/O, u8 spikes, decay 0.5, V_th 1, hard reset,
sigmoid surrogate alpha = 4), with seeded synthetic inputs already resident in HBM.
Prints ONE JSON line: neuron-timesteps/s over the timed steps, the HBM roofline of the
dominant kernel (the backward) from HIP events recorded on the launch stream around every
launch, a plain copy's bandwidth on the box, and -- after the timed region -- the timed
step's outputs checked against the CPU oracle on sampled neurons and the oracle's own
throughput on the host as a baseline (one core pinned, and all cores).

    python bench.py [--steps K] [--warmup W] [--workload conv|single|long|stack|large]
                    [--T T] [--fused-stack | --depth-stack] [--graph-trials N]
                    [--no-cpu-baseline] [--no-configs] [--config-steps K2] [--with-copy]
                    [--compare-serial [--Ts ...]]

The default run (the conv-shaped headline) then also measures every other workload --
the single layer, the long layer, the stack in its three schedules, the large bf16 layer
at T = 4, 16, 64 and 256 -- each with its own timed steps and sampled oracle check, and
records them under "configs" in the same line (--no-configs skips them).

--fused-stack runs a stack's layers after the first fed straight from the previous
layer's spikes through the gain (no stored input current or dL/dx between layers);
--depth-stack runs the whole stack as one kernel per direction.  --graph-trials (single
workload) adds independent forward+backward trials replayed from one HIP graph as a
separate figure; --with-copy adds the 1 GiB copy that calibrates the traffic counters;
--compare-serial times the fused layer against the per-step serial baseline over T.

Workloads whose buffers are smaller than the 256 MB Infinity Cache rotate over several
independent buffer sets (about 1 GiB in total), one set per step, so that a step does not
find the previous step's data in the cache.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, published
KERNEL_SRC_DIR = os.path.join(ROOT, "paper_2408_00280_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")
ROTATE_BYTES = 1 << 30


def bytes_per_nts(w):
    """Algorithmic HBM bytes per neuron-timestep: each I/O tensor read or written once.
    LIF forward: read x, write spikes; LIF backward: read x (recompute) and dL/dy, write
    dL/dx; gain forward: read spikes, write x_next; gain backward: read and write.  The
    gain-fed layer: forward reads the previous spikes and writes its own; backward reads
    the previous spikes and dL/dy, writes dL/d(previous spikes).  The stack fused across
    depth counts per position of the stack, not per layer."""
    e = 4 if w.io == "f32" else 2
    s = 1.0 if w.spk == "u8" else 0.125
    return {"lif_forward": e + s, "lif_backward": 3 * e, "gain_forward": s + e, "gain_backward": 2 * e,
            "lif_forward_gain": 2 * s, "lif_backward_gain": s + 2 * e,
            # the whole stack in one kernel, per position (t, n): x in and the last layer's
            # spikes out; x and the last layer's dL/dy in, the first layer's dL/dx out
            "lif_stack_forward": e + s, "lif_stack_backward": 3 * e}


def code_of(text: str) -> str:
    """C/C++ source without its comments, whitespace runs collapsed: what the compiler sees
    of it, so that editing a comment does not make measurements of the code look stale."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def source_hash(src_dir: str = KERNEL_SRC_DIR) -> str:
    """Hash of the kernel code (every file under csrc/, in name order, comments removed)."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(src_dir)):
        with open(os.path.join(src_dir, name), encoding="utf-8") as f:
            h.update(name.encode() + b"\0" + code_of(f.read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(kernel_tag: str, workload_tag: str):
    """HBM bytes per launch from a committed rocprofv3 PMC summary, if it was taken on the
    current kernel source; else None."""
    path = os.path.join(PROFILES, f"{kernel_tag}_{workload_tag}_pmc.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_src = re.search(r"source_sha256_16:\s*([0-9a-f]+)", text)
    m_val = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not (m_src and m_val) or m_src.group(1) != source_hash():
        return None
    return float(m_val.group(1))


def _oracle_pass(p, x_np, gs_np, gains, F):
    """Forward + backward of the whole step through the CPU oracle."""
    import oracle
    if gains is None:
        y, v = oracle.forward(p, x_np)
        oracle.backward(p, v, y, gs_np)
    else:
        B = x_np.shape[1] // F
        _, ys, vs = oracle.stack_forward(p, x_np, gains, B, F)
        oracle.stack_backward(p, ys, vs, gs_np, gains, B, F)


def host_threads() -> int:
    """Host cores this process may use (the affinity mask, capped by OMP_NUM_THREADS if set)."""
    n = len(os.sched_getaffinity(0))
    cap = os.environ.get("OMP_NUM_THREADS")
    return max(1, min(n, int(cap))) if cap and cap.isdigit() else n


def _repeat(fn, min_s: float = 3.0):
    """Run fn until at least min_s seconds have passed; (seconds per run, runs)."""
    runs, t0 = 0, time.perf_counter()
    while True:
        fn()
        runs += 1
        dt = time.perf_counter() - t0
        if dt >= min_s:
            return dt / runs, runs


def host_info() -> dict:
    """The host CPU and the oracle's compiler and flags."""
    import subprocess

    import oracle
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
    except OSError:
        pass
    try:
        gcc = subprocess.run(["gcc", "--version"], capture_output=True, text=True, timeout=30).stdout.splitlines()[0]
    except (OSError, IndexError, subprocess.SubprocessError):
        gcc = None
    return {"cpu_model": model, "logical_cpus": os.cpu_count(), "threads_allowed": host_threads(),
            "oracle_compiler": gcc, "oracle_cflags": " ".join(oracle.CFLAGS)}


def _pinned_single_core(p, x_np, gs_np, gains, F, reps: int = 3) -> dict:
    """Forward and backward of the oracle timed separately on one thread pinned to one core
    (sched_setaffinity on the calling thread), median of `reps` runs each."""
    import numpy as np

    import oracle
    allowed = sorted(os.sched_getaffinity(0))
    core = allowed[-1]
    os.sched_setaffinity(0, {core})
    try:
        fwd, bwd = [], []
        for _ in range(reps):
            t0 = time.perf_counter()
            if gains is None:
                y, v = oracle.forward(p, x_np)
            else:
                B = x_np.shape[1] // F
                _, ys, vs = oracle.stack_forward(p, x_np, gains, B, F)
            t1 = time.perf_counter()
            if gains is None:
                oracle.backward(p, v, y, gs_np)
            else:
                oracle.stack_backward(p, ys, vs, gs_np, gains, B, F)
            t2 = time.perf_counter()
            fwd.append(t1 - t0)
            bwd.append(t2 - t1)
    finally:
        os.sched_setaffinity(0, set(allowed))
    return {"core": core, "pinned": "sched_setaffinity of the calling thread", "reps": reps,
            "forward_s_median": float(np.median(fwd)), "backward_s_median": float(np.median(bwd)),
            "forward_s": fwd, "backward_s": bwd}


def cpu_baseline(w, x_np, gs_np, gains=None):
    """The CPU oracle on the host: one thread pinned to one core (forward and backward timed
    separately), then the same oracle functions on disjoint neuron slices, one thread per
    core (the slicing is harness code; the oracle releases the interpreter lock inside its
    C calls)."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    p = oracle.Params.of(w.params)
    layers = 1 if gains is None else len(gains) + 1
    T, n = x_np.shape
    nts = layers * T * n
    one = _pinned_single_core(p, x_np, gs_np, gains, w.F)
    dt1 = one["forward_s_median"] + one["backward_s_median"]

    cores = host_threads()
    unit = w.F if gains is not None else 1          # stack slices keep whole feature rows
    groups = n // unit
    bounds = [unit * (groups * i // cores) for i in range(cores + 1)]
    parts = [(np.ascontiguousarray(x_np[:, a:b]), np.ascontiguousarray(gs_np[:, a:b]))
             for a, b in zip(bounds[:-1], bounds[1:]) if b > a]
    with ThreadPoolExecutor(max_workers=len(parts)) as pool:
        dtn, runsn = _repeat(lambda: list(pool.map(lambda xg: _oracle_pass(p, xg[0], xg[1], gains, w.F), parts)))
    what = "the whole workload" if n == w.N else f"the first {n} neurons of {w.N}"
    return {"value": nts / dtn, "unit": "neuron-timesteps/s", "cores": len(parts), "kind": "oracle",
            "sample": f"{layers} layer(s) x {T} steps x {n} neurons ({nts} nts, {what}), forward + backward, "
                      f"{len(parts)} threads on disjoint neuron slices, {runsn} run(s) of {dtn:.3f} s",
            "single_thread": {"value": nts / dt1, "cores": 1, "seconds_per_run": dt1,
                              "forward_nts_per_s": nts / one["forward_s_median"],
                              "backward_nts_per_s": nts / one["backward_s_median"], **one},
            "host": host_info()}


def sample_columns(N: int, n_sample: int = 4096, seed: int = 0):
    """Neuron columns for the parity check: the first and last 1024, plus random ones."""
    import numpy as np
    if N <= n_sample:
        return np.arange(N)
    rng = np.random.default_rng(seed)
    edge = np.r_[np.arange(1024), np.arange(N - 1024, N)]
    inner = 1024 + rng.choice(N - 2048, size=n_sample - edge.size, replace=False)
    return np.unique(np.r_[edge, inner])


def parity_check(w, st, gains_np, schedule: str, cols) -> dict:
    """The timed step's outputs (one buffer set, after the timed region) against the oracle
    on sampled neuron columns: every stored layer's spikes exactly (near-threshold rule) and
    the first layer's dL/dx within the oracle's error budgets (tests/parity.py)."""
    import numpy as np

    import oracle
    from synth import workloads as W
    from tests import gpu_harness, parity
    L = w.layers
    p = oracle.Params.of(w.params)
    x, gs = W.x_cols(w, cols), W.gs_cols(w, cols)
    rep = parity.Report()
    if L == 1:
        y_ref, v_ref = oracle.forward(p, x)
        ys, vs = [y_ref], [v_ref]
        ref = oracle.backward(p, v_ref, y_ref, gs)
    else:
        F = w.F
        g_io = [gpu_harness.round_io(g[cols % F], w.io) for g in gains_np]
        _, ys, vs = oracle.stack_forward(p, x, g_io, 1, cols.size)
        ref = oracle.stack_backward(p, ys, vs, gs, g_io, 1, cols.size)[0]
    stored = [L - 1] if schedule == "fused across depth" else list(range(L))
    g_gpu = None
    for l in stored:   # spikes the schedule stores, and the first layer's dL/dx
        y_gpu, _, g_gpu = gpu_harness.gather_columns(w, st["spk"][l], None, st["g"][0], cols)
        parity.compare_forward(y_gpu, ys[l], vs[l], w.params.v_th, rep=rep)
    parity.compare_grad(g_gpu, ref, w.io, rep)
    return {"ok": rep.ok(), "columns": int(cols.size), "layers_checked": stored, **rep.counts(),
            "rule": "spikes exact unless the oracle membrane is strictly within 1e-5 of V_th; dL/dx within "
                    "q|ref| + (1+q)(1e-5 err + 2^-8 rnd), q = 2^-8 for bf16 storage else 0"}


def copy_ceiling(torch, dev, nbytes: int = 1 << 30, reps: int = 5) -> dict:
    """A plain device-to-device copy of `nbytes`: the practical HBM ceiling on this machine."""
    a = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b
    return {"bytes_copied": nbytes, "ms": ms, "GB/s": 2 * nbytes / (ms * 1e-3) / 1e9,
            "frac_of_peak": 2 * nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "note": "torch copy_ of 1 GiB, read + write bytes over event time"}


def compare_serial(args):
    """Fused vs serial (one launch per step) forward + backward of one layer over a sweep of
    T: the shape of the paper's single-GPU time-step experiment.  One JSON line per T."""
    import torch

    from paper_2408_00280_amd import layer, native
    from synth import workloads as W

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    base = W.WORKLOADS[args.workload if args.workload != "conv" else "paper_monolayer"]
    for T in [int(t) for t in args.Ts.split(",")]:
        w = base.with_T(T)
        N = w.N
        cfg = layer.LifConfig(w.params.decay, w.params.v_th, w.params.v_reset, w.params.alpha,
                              w.params.reset, w.io, w.spk)
        c = cfg.c()
        x = torch.from_numpy(W.x_full(w)).to(dev)
        gs = torch.from_numpy(W.gs_full(w)).to(dev)
        spikes, saved, _ = layer.alloc_forward(cfg, T, N, dev)
        sv = saved if saved.numel() else None
        gx = torch.empty_like(gs)
        v = torch.empty((T, N), dtype=torch.float32, device=dev)

        # launches go to torch's current stream (the capture stream inside a graph capture)
        def fused():
            native.snn_lif_forward(c, T, N, x, spikes, sv, None)
            native.snn_lif_backward(c, T, N, x, sv, gs, gx)

        def serial():
            for t in range(T):
                native.snn_lif_serial_forward_step(c, N, x[t], v[t - 1] if t else None, v[t], spikes[t])
            for t in range(T - 1, -1, -1):
                native.snn_lif_serial_backward_step(c, N, v[t], gs[t], gx[t + 1] if t + 1 < T else None, gx[t])

        def timed(fn, reps):
            for _ in range(3):
                fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / reps

        fused_ms = timed(fused, args.trials)
        serial_ms = timed(serial, args.trials)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            serial()
        graph_ms = timed(g.replay, args.trials)
        # the graph replays must reproduce the eager serial result
        gx_graph = gx.clone()
        serial()
        torch.cuda.synchronize()
        assert torch.equal(gx_graph, gx), "graph replay differs from the eager serial run"
        fused_bytes = (bytes_per_nts(w)["lif_forward"] + bytes_per_nts(w)["lif_backward"]) * T * N
        print(json.dumps({"metric": "fused vs serial LIF forward+backward, ms per trial", "workload": w.description,
                          "T": T, "N": N, "trials": args.trials, "fused_ms": fused_ms, "serial_ms": serial_ms,
                          "serial_graph_ms": graph_ms, "speedup_vs_serial": serial_ms / fused_ms,
                          "speedup_vs_serial_graph": graph_ms / fused_ms,
                          "fused_hbm_fraction": fused_bytes / (fused_ms * 1e-3) / 1e9 / HBM_PEAK_GBS}),
              flush=True)
        del x, gs, spikes, saved, gx, v, g
        torch.cuda.empty_cache()


def system_info(torch) -> dict:
    """The device and software the numbers were taken on."""
    props = torch.cuda.get_device_properties(0)
    rocm = None
    try:
        with open(os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), ".info", "version")) as f:
            rocm = f.read().strip()
    except OSError:
        pass
    return {"device": props.name, "arch": getattr(props, "gcnArchName", None),
            "compute_units": props.multi_processor_count, "hbm_bytes": props.total_memory,
            "rocm": rocm, "hip_runtime": torch.version.hip, "torch": torch.__version__,
            "library_built_with": "hipcc --offload-arch=gfx950 -O3 -ffp-contract=off, packed fp32 off"}


def graph_trials(c, T, N, x0, gs0, row, sbytes, trials, bpn, dev):
    """`trials` independent forward+backward pairs of one layer, captured into one HIP graph
    and replayed (the paper measures its monolayer over 1000 trials).  Each trial has its
    own x, dL/dy and output buffers, up to 1 GiB in total, then they repeat."""
    import torch

    from paper_2408_00280_amd import native
    esz = x0.element_size()
    per = T * N * 3 * esz + T * row + sbytes
    R = max(1, min(trials, ROTATE_BYTES // per))
    bufs = [{"x": x0.clone(), "gs": gs0.clone(), "g": torch.empty_like(gs0),
             "spk": torch.empty((T, row), dtype=torch.uint8, device=dev),
             "saved": torch.empty(sbytes, dtype=torch.uint8, device=dev) if sbytes else None} for _ in range(R)]
    torch.cuda.synchronize()

    def run():
        s = torch.cuda.current_stream().cuda_stream   # the capture stream while capturing
        for i in range(trials):
            b = bufs[i % R]
            native.snn_lif_forward(c, T, N, b["x"], b["spk"], b["saved"], None, s)
            native.snn_lif_backward(c, T, N, b["x"], b["saved"], b["gs"], b["g"], s)

    run()
    eager_g = bufs[0]["g"].clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    for _ in range(2):
        g.replay()
    torch.cuda.synchronize()
    assert torch.equal(bufs[0]["g"], eager_g), "graph replay differs from the eager run"
    reps = 5
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    nbytes = (bpn["lif_forward"] + bpn["lif_backward"]) * T * N * trials
    return {"trials": trials, "buffer_sets": R, "ms_per_replay": ms, "us_per_trial": ms * 1e3 / trials,
            "value": trials * T * N / (ms * 1e-3), "unit": "neuron-timesteps/s",
            "hbm_fraction": nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "note": "forward+backward pairs replayed from one HIP graph; not the per-call figure"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="conv")
    ap.add_argument("--T", type=int, default=None, help="override T (large workload sweep)")
    ap.add_argument("--fused-stack", action="store_true",
                    help="stack: layers after the first read the previous spikes through the gain")
    ap.add_argument("--depth-stack", action="store_true",
                    help="stack: every layer in one kernel per direction (fused across depth)")
    ap.add_argument("--graph-trials", type=int, default=None,
                    help="also time this many independent forward+backward trials replayed from one HIP "
                         "graph (default 1000 for the single workload, else off)")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle leg (the sampled parity check and the CPU baseline)")
    ap.add_argument("--no-configs", action="store_true",
                    help="default run only: skip measuring the other workloads after the headline")
    ap.add_argument("--config-steps", type=int, default=10,
                    help="timed steps for each of the other workloads in the default run")
    ap.add_argument("--with-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration runs)")
    ap.add_argument("--compare-serial", action="store_true",
                    help="fused vs per-step serial forward+backward over --Ts (one JSON line per T)")
    ap.add_argument("--Ts", default="4,8,16,32,64,128,256")
    ap.add_argument("--trials", type=int, default=20)
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the LIF layer shards over neurons with no "
              "communication, so a multi-GPU run is not part of this benchmark", file=sys.stderr)
        sys.exit(2)

    if args.compare_serial:
        compare_serial(args)
        return

    out = measure(args)
    headline = (args.workload == "conv" and args.T is None and not args.fused_stack and not args.depth_stack)
    if headline and not args.no_configs:
        out["configs"] = other_configs(args)
    print(json.dumps(out), flush=True)
    bad = [name for name, rec in [("headline", out)] + list(out.get("configs", {}).items())
           if "parity" in rec and not rec["parity"]["ok"]]
    if bad:
        print(f"bench.py: the timed outputs do not match the oracle ({', '.join(bad)})", file=sys.stderr)
        sys.exit(1)


# The other workloads, measured after the headline in the same default run: each with its
# own timed steps and sampled oracle check (no CPU baseline), so that one run records
# every configuration.
OTHER_CONFIGS = [
    ("single", dict(workload="single")),
    ("long", dict(workload="long")),
    ("stack", dict(workload="stack")),
    ("stack_fused_gain", dict(workload="stack", fused_stack=True)),
    ("stack_fused_depth", dict(workload="stack", depth_stack=True)),
    ("large_T4", dict(workload="large", T=4)),
    ("large_T16", dict(workload="large", T=16)),
    ("large_T64", dict(workload="large", T=64)),
    ("large_T256", dict(workload="large", T=256)),
]


def other_configs(args) -> dict:
    import torch
    keep = ("value", "unit", "ms_per_step", "steps", "warmup", "dtype", "config", "hbm_fraction_step", "roofline",
            "kernels", "parity", "graph_trials")
    res = {}
    for name, over in OTHER_CONFIGS:
        a = argparse.Namespace(**vars(args))
        a.workload, a.T, a.fused_stack, a.depth_stack = over["workload"], over.get("T"), False, False
        a.fused_stack = over.get("fused_stack", False)
        a.depth_stack = over.get("depth_stack", False)
        a.steps, a.warmup, a.with_copy, a.parity_only = args.config_steps, 2, False, True
        a.graph_trials = None
        print(f"bench.py: {name}", file=sys.stderr, flush=True)
        try:
            rec = measure(a)
        except Exception as e:   # recorded; the headline above stands on its own
            res[name] = {"error": f"{type(e).__name__}: {e}"}
            print(f"bench.py: {name} failed: {e}", file=sys.stderr, flush=True)
        else:
            res[name] = {k: rec[k] for k in keep if k in rec}
        torch.cuda.empty_cache()
    return res


def measure(args) -> dict:
    """One workload: warmup, timed steps, the record (and the oracle leg unless skipped)."""
    import numpy as np
    import torch

    import synth
    from paper_2408_00280_amd import layer, native
    from synth import workloads as W

    w = W.WORKLOADS[args.workload]
    if args.T:
        w = w.with_T(args.T)
    dev = torch.device("cuda:0")
    cfg = layer.LifConfig(w.params.decay, w.params.v_th, w.params.v_reset, w.params.alpha,
                          w.params.reset, w.io, w.spk)
    c = cfg.c()
    T, N, L = w.T, w.N, w.layers
    dt = layer.IO_DTYPES[w.io]
    esz = 4 if w.io == "f32" else 2
    B, F = (N // w.F, w.F)

    # seeded inputs, generated on the host in row chunks and copied to HBM
    parity_only = getattr(args, "parity_only", False)
    keep_host = not args.no_cpu_baseline and not parity_only and T * N <= (1 << 28)
    x0 = torch.empty((T, N), dtype=dt, device=dev)
    gs0 = torch.empty((T, N), dtype=dt, device=dev)
    host = {"x": [], "gs": []}
    rows = max(1, (1 << 26) // N)
    for name, gen, dst in (("x", W.x_rows, x0), ("gs", W.gs_rows, gs0)):
        for t0 in range(0, T, rows):
            a = gen(w, t0, min(T, t0 + rows))
            if keep_host:
                host[name].append(a)
            if w.io == "f32":
                dst[t0:t0 + a.shape[0]].copy_(torch.from_numpy(a))
            else:
                bits = synth.to_bf16_bits(a).view(np.int16)
                dst[t0:t0 + a.shape[0]].copy_(torch.from_numpy(bits).view(torch.bfloat16))
    gains_np = [W.gain(w, l) for l in range(L - 1)]
    gains = [torch.from_numpy(g).to(dev) for g in gains_np]

    # buffer sets: x / spikes / checkpoints per layer, one dL/dy-dL/dx pair per layer
    row = native.snn_spike_row_bytes(c, N)
    sbytes = native.snn_lif_saved_bytes(c, T, N)
    set_bytes = L * T * (2 * N * esz + row) + 2 * T * N * esz + L * sbytes
    R = max(1, min(64, -(-ROTATE_BYTES // set_bytes))) if set_bytes < (512 << 20) else 1
    sets = []
    for _ in range(R):
        st = {"x": [x0.clone() if R > 1 else x0] + [torch.empty_like(x0) for _ in range(L - 1)],
              "spk": [torch.empty((T, row), dtype=torch.uint8, device=dev) for _ in range(L)],
              "saved": [torch.empty(sbytes, dtype=torch.uint8, device=dev) if sbytes else None for _ in range(L)],
              "gs": gs0.clone() if R > 1 else gs0,
              "g": [torch.empty_like(gs0) for _ in range(L)]}
        sets.append(st)
    stream = torch.cuda.current_stream()
    s_ptr = stream.cuda_stream
    torch.cuda.synchronize()

    bpn = bytes_per_nts(w)
    nts = T * N

    fused = args.fused_stack and L > 1
    depth = args.depth_stack and L > 1
    if depth:
        gstack = torch.stack(gains).contiguous()
        dsaved = native.snn_lif_stack_saved_bytes(c, L, T, N)
        for st in sets:
            st["dsaved"] = torch.empty(dsaved, dtype=torch.uint8, device=dev) if dsaved else None

    def launches_depth(st):
        return [("lif_stack_forward", bpn["lif_stack_forward"] * nts, lambda: native.snn_lif_stack_forward(
                    c, L, T, B, F, st["x"][0], gstack, st["spk"][L - 1], None, st["dsaved"], None, s_ptr)),
                ("lif_stack_backward", bpn["lif_stack_backward"] * nts, lambda: native.snn_lif_stack_backward(
                    c, L, T, B, F, st["x"][0], gstack, st["dsaved"], st["gs"], st["g"][0], s_ptr))]

    def launches_fused(st):
        out = [("lif_forward", bpn["lif_forward"] * nts, lambda: native.snn_lif_forward(
            c, T, N, st["x"][0], st["spk"][0], st["saved"][0], None, s_ptr))]
        for l in range(1, L):
            out.append(("lif_forward_gain", bpn["lif_forward_gain"] * nts, lambda l=l: native.snn_lif_forward_gain(
                c, T, B, F, st["spk"][l - 1], gains[l - 1], st["spk"][l], st["saved"][l], None, s_ptr)))
        for l in range(L - 1, 0, -1):
            gy = st["gs"] if l == L - 1 else st["g"][l + 1]
            out.append(("lif_backward_gain", bpn["lif_backward_gain"] * nts,
                        lambda l=l, gy=gy: native.snn_lif_backward_gain(
                            c, T, B, F, st["spk"][l - 1], gains[l - 1], st["saved"][l], gy, st["g"][l], s_ptr)))
        gy = st["gs"] if L == 1 else st["g"][1]
        out.append(("lif_backward", bpn["lif_backward"] * nts, lambda: native.snn_lif_backward(
            c, T, N, st["x"][0], st["saved"][0], gy, st["g"][0], s_ptr)))
        return out

    def launches(st):
        """The kernels of one step, in order: (kernel, algorithmic bytes, call)."""
        if depth:
            return launches_depth(st)
        if fused:
            return launches_fused(st)
        out = []
        for l in range(L):
            out.append(("lif_forward", bpn["lif_forward"] * nts, lambda l=l: native.snn_lif_forward(
                c, T, N, st["x"][l], st["spk"][l], st["saved"][l], None, s_ptr)))
            if l + 1 < L:
                out.append(("gain_forward", bpn["gain_forward"] * nts, lambda l=l: native.snn_gain_spikes_forward(
                    c, T, B, F, st["spk"][l], gains[l], st["x"][l + 1], s_ptr)))
        for l in range(L - 1, -1, -1):
            gy = st["gs"] if l == L - 1 else st["g"][l + 1]   # gain backward writes in place
            out.append(("lif_backward", bpn["lif_backward"] * nts, lambda l=l, gy=gy: native.snn_lif_backward(
                c, T, N, st["x"][l], st["saved"][l], gy, st["g"][l], s_ptr)))
            if l > 0:
                out.append(("gain_backward", bpn["gain_backward"] * nts, lambda l=l: native.snn_gain_grad_backward(
                    c, T, B, F, st["g"][l], gains[l - 1], st["g"][l], s_ptr)))
        return out

    plans = [launches(st) for st in sets]
    n_launch = len(plans[0])

    for i in range(args.warmup):
        for _, _, f in plans[i % R]:
            f()
    torch.cuda.synchronize()

    K = args.steps
    # one event before the first launch and one after every launch: launch j of step i runs
    # between events i*n_launch + j and the next one
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_launch * K + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(K):
        base = i * n_launch
        for j, (_, _, f) in enumerate(plans[i % R]):
            f()
            ev[base + j + 1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    per = {}
    for i in range(K):
        base = i * n_launch
        for j, (name, nbytes, _) in enumerate(plans[0]):
            d = per.setdefault(name, {"ms": [], "bytes": nbytes})
            d["ms"].append(ev[base + j].elapsed_time(ev[base + j + 1]))
    kernels = {}
    for name, d in per.items():
        ms = float(np.mean(d["ms"]))
        kernels[name + "_kernel"] = {"avg_launch_ms": ms, "median_launch_ms": float(np.median(d["ms"])),
                                     "launches_per_step": len(d["ms"]) // K,
                                     "GB/s": d["bytes"] / (ms * 1e-3) / 1e9,
                                     "bytes_per_nts": bpn[name]}
    step_kernel_ms = sum(v["avg_launch_ms"] * v["launches_per_step"] for v in kernels.values())
    step_bytes = sum(d["bytes"] * len(d["ms"]) / K for d in per.values())

    if args.with_copy:   # counter calibration: a plain copy of known size
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()

    wtag = f"{w.name}{'depth' if depth else 'fused' if fused else ''}_T{T}_N{N}"
    # the dominant kernel: the largest share of the step's kernel time
    dom_name = max(kernels, key=lambda k: kernels[k]["avg_launch_ms"] * kernels[k]["launches_per_step"])
    dom = kernels[dom_name]
    for name in kernels:
        kernels[name]["traffic"] = measured_traffic(name.replace("_kernel", ""), wtag)
    out = {
        "metric": "neuron-timesteps/sec (LIF fwd+bwd) and % of MI355X HBM peak",
        "value": L * nts * K / elapsed,
        "unit": "neuron-timesteps/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": elapsed / K * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.io == "f32" else "bf16 I/O, f32 compute",
        "data": "synthetic (seeded counter-based generator)",
        "config": {"workload": w.description, "T": T, "N": N, "layers": L, "dims": list(w.dims), "io": w.io,
                   "spikes": w.spk, "reset": w.params.reset, "decay": w.params.decay,
                   "v_th": w.params.v_th, "alpha": w.params.alpha, "buffer_sets": R,
                   "schedule": ("fused across depth" if depth else "fused across the gain" if fused
                                else "layer by layer"),
                   "parallelism": "none (1 GPU)"},
        "hbm_fraction_step": step_bytes / (step_kernel_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "roofline": {"kernel": dom_name, "bound": "hbm", "achieved": dom["GB/s"],
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": dom["GB/s"] / HBM_PEAK_GBS,
                     "traffic": dom["traffic"], "algorithmic_bytes_per_launch": dom["bytes_per_nts"] * nts,
                     "bytes_per_nts": dom["bytes_per_nts"], "avg_launch_ms": dom["avg_launch_ms"]},
        "kernels": kernels,
        "kernel_source_sha256_16": source_hash(),
        "system": system_info(torch),
    }
    trials = args.graph_trials if args.graph_trials is not None else (1000 if w.name == "single" else 0)
    if trials and L == 1:
        out["graph_trials"] = graph_trials(c, T, N, x0, gs0, row, sbytes, trials, bpn, dev)
    if not parity_only:
        out["copy_ceiling"] = copy_ceiling(torch, dev)
    if not args.no_cpu_baseline:
        # the oracle's leg, after the timed region: the timed step's outputs against the
        # oracle on sampled columns, then the oracle's own throughput on the host
        out["parity"] = parity_check(w, sets[(K - 1) % R], gains_np, out["config"]["schedule"],
                                     sample_columns(N))
    if not args.no_cpu_baseline and not parity_only:
        if keep_host:
            x_np, gs_np = np.concatenate(host["x"]), np.concatenate(host["gs"])
        else:   # a bounded sample: the first neurons over all steps
            cols = np.arange(min(N, max(1 << 12, (1 << 28) // T)))
            x_np, gs_np = W.x_cols(w, cols), W.gs_cols(w, cols)
        out["cpu_baseline"] = cpu_baseline(w, x_np, gs_np, gains_np if L > 1 else None)
    return out


if __name__ == "__main__":
    main()
