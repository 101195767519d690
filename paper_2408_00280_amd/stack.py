"""A stack of LIF layers joined by a per-feature gain (a diagonal synapse standing in for
the ANN operator between spiking layers), run layer by layer in temporal-major order:
each layer's fused kernel covers all T steps before the next layer starts (Sec. 3.2).

Three schedules:
  * unfused -- gain kernels between the layers materialise every layer's input current
    x and, in the backward, every layer's dL/dx;
  * fused   -- layers after the first read the previous layer's spikes and the gain
    directly (snn_lif_forward_gain), and their backward emits dL/d(previous spikes)
    (snn_lif_backward_gain); no x or dL/dx beyond the first layer's is stored;
  * depth   -- one kernel per direction runs every layer (snn_lif_stack_forward /
    backward, 2 or 3 layers): only x, the last layer's spikes, the checkpoints and dL/dx
    of the first layer go through memory.
All give the same spikes and membranes bit for bit.

Torch allocates; every step runs in the HIP kernels behind the C ABI.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import layer, native


@dataclass
class LayerState:
    x: torch.Tensor | None   # this layer's input current [T][N] (None when fed through the gain)
    spikes: torch.Tensor     # [T][row_bytes]
    saved: torch.Tensor      # checkpoints
    v: torch.Tensor | None   # optional membrane output


def forward(cfg: layer.LifConfig, x1: torch.Tensor, gains: list[torch.Tensor], B: int, F: int, *,
            v_out: bool = False, fused: bool = False, stream=None) -> list[LayerState]:
    T = x1.shape[0]
    states = []
    x = x1
    for l in range(len(gains) + 1):
        if l > 0 and fused:
            spikes, saved, v = layer.forward_gain(cfg, states[-1].spikes, gains[l - 1], B, F, v_out=v_out,
                                                  stream=stream)
            states.append(LayerState(None, spikes, saved, v))
            continue
        spikes, saved, v = layer.forward(cfg, x, v_out=v_out, stream=stream)
        states.append(LayerState(x, spikes, saved, v))
        if l < len(gains) and not fused:
            x_next = torch.empty_like(x1)
            native.snn_gain_spikes_forward(cfg.c(), T, B, F, spikes, gains[l], x_next, stream)
            x = x_next
    return states


def forward_depth(cfg: layer.LifConfig, x1: torch.Tensor, gains: list[torch.Tensor], B: int, F: int, *,
                  hidden: bool = False, v_out: bool = False, stream=None):
    """The whole stack in one forward kernel.  Returns (spikes of the last layer, hidden
    spikes or None, saved, membranes or None, the stacked gains to pass to the backward)."""
    g = torch.stack([t.to(torch.float32) for t in gains]).contiguous()
    spikes, hid, saved, v = layer.stack_forward(cfg, x1, g, B, F, hidden=hidden, v_out=v_out, stream=stream)
    return spikes, hid, saved, v, g


def backward_depth(cfg: layer.LifConfig, x1: torch.Tensor, g: torch.Tensor, saved: torch.Tensor,
                   grad_s_last: torch.Tensor, B: int, F: int, *, stream=None) -> torch.Tensor:
    """dL/dx of the first layer from dL/dy of the last, in one backward kernel."""
    return layer.stack_backward(cfg, x1, g, saved, grad_s_last, B, F, stream=stream)


def backward(cfg: layer.LifConfig, states: list[LayerState], grad_s_last: torch.Tensor,
             gains: list[torch.Tensor], B: int, F: int, *, stream=None) -> list[torch.Tensor]:
    """Gradients of the stack, first layer first.  Unfused states (every x kept): dL/dx of
    every layer.  Fused states: dL/dx1 of the first layer, then dL/dy of layers 0 .. L-2
    (the gradient each gain-fed layer passes to the spikes that feed it)."""
    T = grad_s_last.shape[0]
    L = len(states)
    if L > 1 and states[1].x is None:
        gys = [None] * (L - 1)
        gy = grad_s_last
        for l in range(L - 1, 0, -1):
            st = states[l]
            gy = layer.backward_gain(cfg, states[l - 1].spikes, gains[l - 1], st.saved, gy, B, F, stream=stream)
            gys[l - 1] = gy
        return [layer.backward(cfg, states[0].x, states[0].saved, gy, stream=stream)] + gys
    grads = [None] * L
    gy = grad_s_last
    for l in range(L - 1, -1, -1):
        st = states[l]
        grads[l] = layer.backward(cfg, st.x, st.saved, gy, stream=stream)
        if l > 0:
            gy = torch.empty_like(grads[l])
            native.snn_gain_grad_backward(cfg.c(), T, B, F, grads[l], gains[l - 1], gy, stream)
    return grads
