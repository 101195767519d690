#!/usr/bin/env python3
"""Benchmark of the temporally fused LIF layer on one MI355X.

One step = the fused forward plus the fused backward of the conv-shaped LIF layer
x[T=16, B=64, C=128, H=32, W=32] (fp32 I/O, u8 spikes, decay 0.5, V_th 1, hard reset,
sigmoid surrogate alpha = 4), with seeded synthetic inputs already resident in HBM.
Prints ONE JSON line: neuron-timesteps/s over the timed steps, the HBM roofline of the
dominant kernel (the backward) from HIP events recorded on the launch stream, and the CPU
oracle's throughput on the host as a baseline.

    python bench.py [--steps K] [--warmup W] [--workload conv|single|long|stack|large]
                    [--T T] [--no-cpu-baseline] [--with-copy]
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
KERNEL_SRC = os.path.join(ROOT, "paper_2408_00280_amd", "csrc", "snn_lif.hip")
PROFILES = os.path.join(ROOT, "profiles")


def bytes_per_nts(w, layers: int = 1):
    """Algorithmic HBM bytes per neuron-timestep: each I/O tensor read or written once.
    forward: read x, write spikes; backward: read x (recompute) and dL/dy, write dL/dx."""
    e = 4 if w.io == "f32" else 2
    s = 1.0 if w.spk == "u8" else 0.125
    return {"forward": e + s, "backward": 3 * e}


def source_hash() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


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


def cpu_baseline(w, x_np, gs_np):
    """The CPU oracle, single-threaded, on the same inputs (forward + backward)."""
    import oracle
    p = oracle.Params.of(w.params)
    t0 = time.perf_counter()
    y, v = oracle.forward(p, x_np)
    oracle.backward(p, v, y, gs_np)
    dt = time.perf_counter() - t0
    nts = x_np.shape[0] * x_np.shape[1]
    return {"value": nts / dt, "unit": "neuron-timesteps/s", "cores": 1, "kind": "oracle",
            "sample": f"whole workload: {x_np.shape[0]} steps x {x_np.shape[1]} neurons "
                      f"({nts} nts), forward + backward, {dt:.2f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="conv")
    ap.add_argument("--T", type=int, default=None, help="override T (large workload sweep)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--with-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration runs)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the LIF layer shards over neurons with no "
              "communication, so a multi-GPU run is not part of this benchmark", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2408_00280_amd import layer
    from synth import workloads as W

    w = W.WORKLOADS[args.workload]
    if args.T:
        w = w.with_T(args.T)
    if w.layers != 1:
        sys.exit("bench.py times single-layer workloads; the stack is covered by the tests")
    dev = torch.device("cuda:0")
    cfg = layer.LifConfig(w.params.decay, w.params.v_th, w.params.v_reset, w.params.alpha,
                          w.params.reset, w.io, w.spk)
    T, N = w.T, w.N
    dt = layer.IO_DTYPES[w.io]

    # seeded inputs, generated on the host in row chunks and copied to HBM
    keep_host = not args.no_cpu_baseline and T * N <= (1 << 28)
    x = torch.empty((T, N), dtype=dt, device=dev)
    gs = torch.empty((T, N), dtype=dt, device=dev)
    host = {"x": [], "gs": []}
    rows = max(1, (1 << 26) // N)
    import synth
    for name, gen, dst in (("x", W.x_rows, x), ("gs", W.gs_rows, gs)):
        for t0 in range(0, T, rows):
            a = gen(w, t0, min(T, t0 + rows))
            if keep_host:
                host[name].append(a)
            if w.io == "f32":
                dst[t0:t0 + a.shape[0]].copy_(torch.from_numpy(a))
            else:
                bits = synth.to_bf16_bits(a).view(np.int16)
                dst[t0:t0 + a.shape[0]].copy_(torch.from_numpy(bits).view(torch.bfloat16))
    spikes, saved, _ = layer.alloc_forward(cfg, T, N, dev)
    gx = torch.empty_like(gs)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    def step(ev=None, i=0):
        if ev is not None:
            ev[3 * i].record(stream)
        layer.forward(cfg, x, out=(spikes, saved, None), stream=stream)
        if ev is not None:
            ev[3 * i + 1].record(stream)
        layer.backward(cfg, x, saved, gs, grad_x=gx, stream=stream)
        if ev is not None:
            ev[3 * i + 2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    K = args.steps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3 * K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        step(ev, i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    fwd_ms = float(np.mean([ev[3 * i].elapsed_time(ev[3 * i + 1]) for i in range(K)]))
    bwd_ms = float(np.mean([ev[3 * i + 1].elapsed_time(ev[3 * i + 2]) for i in range(K)]))

    if args.with_copy:   # counter calibration: a plain copy of known size
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()

    nts = T * N
    bpn = bytes_per_nts(w)
    bwd_bytes = bpn["backward"] * nts
    fwd_bytes = bpn["forward"] * nts
    bwd_gbs = bwd_bytes / (bwd_ms * 1e-3) / 1e9
    fwd_gbs = fwd_bytes / (fwd_ms * 1e-3) / 1e9
    wtag = f"{w.name}_T{T}_N{N}"
    traffic = measured_traffic("lif_backward", wtag)

    out = {
        "metric": "neuron-timesteps/sec (LIF fwd+bwd) and % of MI355X HBM peak",
        "value": nts * K / elapsed,
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
        "config": {"workload": w.description, "T": T, "N": N, "dims": list(w.dims), "io": w.io,
                   "spikes": w.spk, "reset": w.params.reset, "decay": w.params.decay,
                   "v_th": w.params.v_th, "alpha": w.params.alpha, "parallelism": "none (1 GPU)"},
        "hbm_fraction_fwd_bwd": (fwd_bytes + bwd_bytes) / ((fwd_ms + bwd_ms) * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "roofline": {"kernel": "lif_backward_kernel", "bound": "hbm", "achieved": bwd_gbs,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": bwd_gbs / HBM_PEAK_GBS,
                     "traffic": traffic, "algorithmic_bytes_per_launch": bwd_bytes,
                     "bytes_per_nts": bpn["backward"], "avg_launch_ms": bwd_ms},
        "kernels": {"lif_forward_kernel": {"avg_launch_ms": fwd_ms, "GB/s": fwd_gbs,
                                           "bytes_per_nts": bpn["forward"],
                                           "traffic": measured_traffic("lif_forward", wtag)},
                    "lif_backward_kernel": {"avg_launch_ms": bwd_ms, "GB/s": bwd_gbs,
                                            "bytes_per_nts": bpn["backward"]}},
        "kernel_source_sha256_16": source_hash(),
    }
    if not args.no_cpu_baseline:
        if keep_host:
            x_np, gs_np = np.concatenate(host["x"]), np.concatenate(host["gs"])
        else:   # a bounded sample: the first 2^20 neurons over all steps
            cols = np.arange(min(N, 1 << 20))
            x_np, gs_np = W.x_cols(w, cols), W.gs_cols(w, cols)
        out["cpu_baseline"] = cpu_baseline(w, x_np, gs_np)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
