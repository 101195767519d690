"""Helpers for the GPU parity tests: upload seeded inputs, run the HIP path through the
C ABI, run the CPU oracle on the same inputs (all neurons or a sample), compare."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import synth
from paper_2408_00280_amd import layer, native
from synth import workloads as W
from tests import parity

DEV = torch.device("cuda:0")


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def cfg_of(w: W.Workload) -> layer.LifConfig:
    p = w.params
    return layer.LifConfig(p.decay, p.v_th, p.v_reset, p.alpha, p.reset, w.io, w.spk)


def to_dev(a: np.ndarray, io: str) -> torch.Tensor:
    """float32 values (exact in the io dtype) -> device tensor of the io dtype."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if io == "f32":
        return torch.from_numpy(a).to(DEV)
    bits = synth.to_bf16_bits(a)
    return torch.from_numpy(bits.view(np.int16)).to(DEV).view(torch.bfloat16)


def to_host_f32(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return parity.bf16_to_f32(t.view(torch.int16).cpu().numpy())
    return t.float().cpu().numpy()


def upload_rows(w: W.Workload, which: str, rows_per_chunk: int | None = None) -> torch.Tensor:
    """Generate a [T][N] input ("x" or "gs") in row chunks straight into device memory."""
    dt = layer.IO_DTYPES[w.io]
    out = torch.empty((w.T, w.N), dtype=dt, device=DEV)
    rows_per_chunk = rows_per_chunk or max(1, (1 << 26) // max(w.N, 1))
    gen = W.x_rows if which == "x" else W.gs_rows
    big = w.T * w.N >= (1 << 30)
    for t0 in range(0, w.T, rows_per_chunk):
        t1 = min(w.T, t0 + rows_per_chunk)
        out[t0:t1].copy_(to_dev(gen(w, t0, t1), w.io))
        if big and (t0 // rows_per_chunk) % 8 == 0:
            say(f"  {which}: generated rows [0, {t1}) of {w.T}")
    return out


def sample_columns(N: int, n_sample: int, seed: int = 0) -> np.ndarray:
    """Neuron columns to check at full size: the first and last 1024, plus random ones."""
    if N <= n_sample:
        return np.arange(N)
    rng = np.random.default_rng(seed)
    edge = np.r_[np.arange(min(1024, N)), np.arange(max(0, N - 1024), N)]
    rest = rng.choice(N, size=n_sample - edge.size, replace=False)
    return np.unique(np.r_[edge, rest])


def gpu_layer(w: W.Workload, x: torch.Tensor, gs: torch.Tensor, *, v_out=True, inplace=False):
    cfg = cfg_of(w)
    spikes, saved, v = layer.forward(cfg, x, v_out=v_out)
    gx = layer.backward(cfg, x, saved, gs, grad_x=gs if inplace else None)
    torch.cuda.synchronize()
    return spikes, v, gx


def compare_layer(w, spikes, v, gx, x_np, gs_np, cols=None, rep=None):
    """Oracle on x_np/gs_np (columns `cols` of the full problem if given) vs GPU outputs.
    Returns the report and the oracle's (y, v, Grad)."""
    for a, name in ((x_np, "x"), (gs_np, "dL/dy")):   # the oracle must see what the kernel reads
        assert np.array_equal(round_io(a, w.io), np.asarray(a, dtype=np.float32), equal_nan=True), \
            f"{name} is not exact in {w.io}: round it before uploading and before the oracle"
    p = oracle.Params.of(w.params)
    y_ref, v_ref = oracle.forward(p, x_np)
    ref = oracle.backward(p, v_ref, y_ref, gs_np)
    if cols is not None and w.T * w.N > (1 << 31):
        # a layer too large to copy whole: gather the sampled columns on the device
        y_gpu, v_gpu, g_gpu = gather_columns(w, spikes, v, gx, cols)
    else:
        y_gpu = parity.unpack_spikes(to_host_f32(spikes) if w.spk == "io" else spikes.cpu().numpy(), w.N, w.spk)
        v_gpu = None if v is None else v.cpu().numpy()
        g_gpu = to_host_f32(gx)
        if cols is not None:
            y_gpu = y_gpu[:, cols]
            v_gpu = None if v_gpu is None else v_gpu[:, cols]
            g_gpu = g_gpu[:, cols]
    rep = parity.compare_forward(y_gpu, y_ref, v_ref, w.params.v_th, v_gpu=v_gpu, rep=rep)
    parity.compare_grad(g_gpu, ref, w.io, rep)
    return rep, (y_ref, v_ref, ref)


def gather_columns(w: W.Workload, spikes, v, gx, cols: np.ndarray):
    """Spikes (0/1), membranes and dL/dx of neuron columns `cols`, gathered on the device."""
    c = torch.from_numpy(np.asarray(cols, dtype=np.int64)).to(DEV)
    if w.spk == "io":
        y = to_host_f32(spikes.index_select(1, c)).astype(np.uint8)
    elif w.spk == "u8":
        y = spikes.index_select(1, c).cpu().numpy()
    else:
        byte = spikes.index_select(1, c >> 3).to(torch.int32)
        y = ((byte >> (c & 7).to(torch.int32)) & 1).to(torch.uint8).cpu().numpy()
    vv = None if v is None else v.index_select(1, c).cpu().numpy()
    return y, vv, to_host_f32(gx.index_select(1, c))


def check_full(w: W.Workload, *, v_out=True, inplace=False):
    """Whole problem on both sides."""
    x_np, gs_np = W.x_full(w), W.gs_full(w)
    spikes, v, gx = gpu_layer(w, to_dev(x_np, w.io), to_dev(gs_np, w.io), v_out=v_out, inplace=inplace)
    rep, _ = compare_layer(w, spikes, v, gx, x_np, gs_np)
    return rep


def check_sampled(w: W.Workload, n_sample: int, *, v_out=False):
    """Whole problem on the GPU (generated in chunks on the host), oracle on sampled columns."""
    x = upload_rows(w, "x")
    gs = upload_rows(w, "gs")
    spikes, v, gx = gpu_layer(w, x, gs, v_out=v_out)
    del x, gs
    cols = sample_columns(w.N, n_sample)
    rep, _ = compare_layer(w, spikes, v, gx, W.x_cols(w, cols), W.gs_cols(w, cols), cols=cols)
    return rep


def synth_bf16(a: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (round to nearest even), from the input generator module."""
    return synth.to_bf16_bits(a)


def round_io(a: np.ndarray, io: str) -> np.ndarray:
    """float32 values rounded to the I/O dtype (to nearest even for bf16), as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return parity.bf16_to_f32(synth.to_bf16_bits(a)) if io == "bf16" else a


__all__ = ["DEV", "say", "cfg_of", "to_dev", "to_host_f32", "upload_rows", "sample_columns", "gpu_layer",
           "compare_layer", "gather_columns", "check_full", "check_sampled", "synth_bf16", "round_io", "layer", "native", "np", "torch", "W",
           "oracle", "parity"]
