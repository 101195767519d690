"""The serial (per-time-step) training method, as an ablation baseline for temporal fusion.

One kernel launch per time step and direction, with the fp32 membrane (forward) and the
fp32 dL/dv (backward) round-tripping through memory between steps -- the pattern the paper
contrasts with temporal fusion (Sec. 3.2, Fig. 3).  Results equal the fused path's.
"""
from __future__ import annotations

import torch

from . import layer, native


def forward(cfg: layer.LifConfig, x: torch.Tensor, *, stream=None):
    """x[T][N] -> (spikes in cfg.spk format, v[T][N] fp32 membranes kept for the backward)."""
    if x.dtype != cfg.dtype or not x.is_contiguous():
        raise ValueError(f"x must be a contiguous {cfg.dtype} tensor")
    T = x.shape[0]
    N = x.numel() // T if T else 0
    spikes, _, _ = layer.alloc_forward(cfg, T, N, x.device)
    v = torch.empty((T, N), dtype=torch.float32, device=x.device)
    c = cfg.c()
    x2 = x.view(T, N)
    for t in range(T):
        native.snn_lif_serial_forward_step(c, N, x2[t], v[t - 1] if t else None, v[t], spikes[t], stream)
    return spikes, v


def backward(cfg: layer.LifConfig, v: torch.Tensor, grad_s: torch.Tensor, *, stream=None) -> torch.Tensor:
    """v[T][N] from forward(), dL/dy[T][N] -> dL/dx[T][N] (I/O dtype)."""
    T, N = v.shape
    gs = grad_s.contiguous().view(T, N)
    gx = torch.empty_like(gs)
    c = cfg.c()
    if cfg.io == "f32":        # dL/dx in fp32 is also the state for the previous step
        for t in range(T - 1, -1, -1):
            native.snn_lif_serial_backward_step(c, N, v[t], gs[t], gx[t + 1] if t + 1 < T else None, gx[t],
                                                None, stream)
    else:
        g = torch.empty((2, N), dtype=torch.float32, device=v.device)
        for t in range(T - 1, -1, -1):
            native.snn_lif_serial_backward_step(c, N, v[t], gs[t], g[(t + 1) % 2] if t + 1 < T else None, gx[t],
                                                g[t % 2], stream)
    return gx.view(grad_s.shape)
