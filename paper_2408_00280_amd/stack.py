"""A stack of LIF layers joined by a per-feature gain (a diagonal synapse standing in for
the ANN operator between spiking layers), run layer by layer in temporal-major order:
each layer's fused kernel covers all T steps before the next layer starts (Sec. 3.2).

Torch allocates; every step runs in the HIP kernels behind the C ABI.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import layer, native


@dataclass
class LayerState:
    x: torch.Tensor          # this layer's input current [T][N] (kept for the backward)
    spikes: torch.Tensor     # [T][row_bytes]
    saved: torch.Tensor      # checkpoints
    v: torch.Tensor | None   # optional membrane output


def forward(cfg: layer.LifConfig, x1: torch.Tensor, gains: list[torch.Tensor], B: int, F: int, *,
            v_out: bool = False, stream=None) -> list[LayerState]:
    T = x1.shape[0]
    states = []
    x = x1
    for l in range(len(gains) + 1):
        spikes, saved, v = layer.forward(cfg, x, v_out=v_out, stream=stream)
        states.append(LayerState(x, spikes, saved, v))
        if l < len(gains):
            x_next = torch.empty_like(x1)
            native.snn_gain_spikes_forward(cfg.c(), T, B, F, spikes, gains[l], x_next, stream)
            x = x_next
    return states


def backward(cfg: layer.LifConfig, states: list[LayerState], grad_s_last: torch.Tensor,
             gains: list[torch.Tensor], B: int, F: int, *, stream=None) -> list[torch.Tensor]:
    """dL/dx of every layer, first layer first.  Buffers are reused in place where safe."""
    T = grad_s_last.shape[0]
    L = len(states)
    grads = [None] * L
    gy = grad_s_last
    for l in range(L - 1, -1, -1):
        st = states[l]
        grads[l] = layer.backward(cfg, st.x, st.saved, gy, stream=stream)
        if l > 0:
            gy = torch.empty_like(grads[l])
            native.snn_gain_grad_backward(cfg.c(), T, B, F, grads[l], gains[l - 1], gy, stream)
    return grads
