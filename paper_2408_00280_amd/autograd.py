"""The fused LIF layer as a torch autograd function and module.

This is the programming model of the paper's Listing 1 (a ``FusedLIF`` autograd function
wrapping the fused forward and backward kernels, and a ``LIFLayer`` module to drop into
``torch.nn.Sequential`` next to ANN operators), with two differences: the state the
backward needs (the input current and the membrane checkpoints) is saved explicitly, and
the backward returns no gradient for the hyper-parameters.

Inputs are time-major, ``x[T, ...]``, float32 or bfloat16; the output is the spike train
``y[T, ...]`` as 0/1 values of the same dtype.  The arithmetic runs in the HIP kernels;
torch allocates and orders the work on its current stream.
"""
from __future__ import annotations

import torch

from . import layer

_IO = {torch.float32: "f32", torch.bfloat16: "bf16"}


class FusedLIF(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x: torch.Tensor, cfg: layer.LifConfig):
        if x.dtype not in _IO or cfg.io != _IO[x.dtype] or cfg.spk != "io":
            raise TypeError("FusedLIF takes float32/bfloat16 input and a cfg with io matching it and spk='io'")
        xc = x.contiguous()
        T = xc.shape[0]
        x2 = xc.view(T, -1)
        spikes, saved, _ = layer.forward(cfg, x2)
        ctx.save_for_backward(x2, saved)
        ctx.cfg = cfg
        ctx.shape = x.shape
        return spikes.view(x.shape)

    @staticmethod
    def backward(ctx, grad_y: torch.Tensor):
        x2, saved = ctx.saved_tensors
        g = grad_y.to(x2.dtype).contiguous().view(x2.shape)
        grad_x = layer.backward(ctx.cfg, x2, saved, g)
        return grad_x.view(ctx.shape), None


class LIFLayer(torch.nn.Module):
    """Leaky integrate-and-fire neurons over the leading (time) axis of the input.

    decay is k_tau of Eq. (1) (k_tau = 1 - 1/tau), v_th the threshold of Eq. (2), v_reset
    V_rest (initial membrane and hard-reset value), alpha the sigmoid-surrogate sharpness,
    reset "hard" (Eq. (1)) or "soft" (subtract the threshold)."""

    def __init__(self, decay: float, v_th: float, v_reset: float = 0.0, alpha: float = 4.0, reset: str = "hard"):
        super().__init__()
        self.decay, self.v_th, self.v_reset, self.alpha, self.reset = decay, v_th, v_reset, alpha, reset

    def cfg(self, dtype: torch.dtype) -> layer.LifConfig:
        return layer.LifConfig(self.decay, self.v_th, self.v_reset, self.alpha, self.reset, _IO[dtype], "io")

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        return FusedLIF.apply(x, self.cfg(x.dtype))

    def extra_repr(self) -> str:
        return (f"decay={self.decay}, v_th={self.v_th}, v_reset={self.v_reset}, alpha={self.alpha}, "
                f"reset={self.reset}")


class FusedGainLIF(torch.autograd.Function):
    """A LIF layer fed by the previous layer's spikes through a fixed per-feature gain:
    input current gain[f] * spikes_in[t, ..., f], formed inside the fused kernels (the gain
    rounded to the I/O dtype first).  The backward returns dL/d spikes_in = gain[f] * dL/dx
    with the same rounded gain; the gain gets no gradient."""

    @staticmethod
    def forward(ctx, spikes_in: torch.Tensor, gain: torch.Tensor, cfg: layer.LifConfig):
        if spikes_in.dtype not in _IO or cfg.io != _IO[spikes_in.dtype] or cfg.spk != "io":
            raise TypeError("FusedGainLIF takes float32/bfloat16 spikes and a cfg with io matching them and spk='io'")
        F = gain.numel()
        if spikes_in.shape[-1] != F or gain.dtype != torch.float32:
            raise ValueError("gain must be float32 with one entry per feature (the last axis of spikes_in)")
        s = spikes_in.contiguous()
        T = s.shape[0]
        B = s.numel() // (T * F) if T else 0
        s2 = s.view(T, B * F)
        g = gain.contiguous()
        spikes, saved, _ = layer.forward_gain(cfg, s2, g, B, F)
        ctx.save_for_backward(s2, g, saved)
        ctx.cfg, ctx.shape, ctx.BF = cfg, spikes_in.shape, (B, F)
        return spikes.view(spikes_in.shape)

    @staticmethod
    def backward(ctx, grad_y: torch.Tensor):
        s2, g, saved = ctx.saved_tensors
        B, F = ctx.BF
        gy = grad_y.to(s2.dtype).contiguous().view(s2.shape)
        grad_in = layer.backward_gain(ctx.cfg, s2, g, saved, gy, B, F)
        return grad_in.view(ctx.shape), None, None


class GainLIF(torch.nn.Module):
    """LIF neurons fed by spikes through a fixed per-feature gain (the feature axis is the
    last one): the fused form of ``x = gain * spikes`` followed by a :class:`LIFLayer`, with
    the same spikes and membranes and without storing x."""

    def __init__(self, gain: torch.Tensor, decay: float, v_th: float, v_reset: float = 0.0, alpha: float = 4.0,
                 reset: str = "hard"):
        super().__init__()
        self.register_buffer("gain", gain.detach().to(torch.float32).contiguous())
        self.decay, self.v_th, self.v_reset, self.alpha, self.reset = decay, v_th, v_reset, alpha, reset

    def cfg(self, dtype: torch.dtype) -> layer.LifConfig:
        return layer.LifConfig(self.decay, self.v_th, self.v_reset, self.alpha, self.reset, _IO[dtype], "io")

    def forward(self, spikes_in: torch.Tensor) -> torch.Tensor:
        return FusedGainLIF.apply(spikes_in, self.gain, self.cfg(spikes_in.dtype))

    def extra_repr(self) -> str:
        return (f"features={self.gain.numel()}, decay={self.decay}, v_th={self.v_th}, v_reset={self.v_reset}, "
                f"alpha={self.alpha}, reset={self.reset}")


class FusedLIFStack(torch.autograd.Function):
    """len(gains) + 1 LIF layers joined by fixed per-feature gains, fused across depth and
    time: one kernel per direction for the whole stack.  Returns the last layer's spikes;
    the backward returns dL/dx of the first layer (the gains get no gradient)."""

    @staticmethod
    def forward(ctx, x: torch.Tensor, gains: torch.Tensor, cfg: layer.LifConfig):
        if x.dtype not in _IO or cfg.io != _IO[x.dtype] or cfg.spk != "io":
            raise TypeError("FusedLIFStack takes float32/bfloat16 input and a cfg with io matching it and spk='io'")
        F = gains.shape[1]
        if x.shape[-1] != F:
            raise ValueError("gains must have one column per feature (the last axis of x)")
        xc = x.contiguous()
        T = xc.shape[0]
        B = xc.numel() // (T * F) if T else 0
        x2 = xc.view(T, B * F)
        g = gains.to(torch.float32).contiguous()
        spikes, _, saved, _ = layer.stack_forward(cfg, x2, g, B, F)
        ctx.save_for_backward(x2, g, saved)
        ctx.cfg, ctx.shape, ctx.BF = cfg, x.shape, (B, F)
        return spikes.view(x.shape)

    @staticmethod
    def backward(ctx, grad_y: torch.Tensor):
        x2, g, saved = ctx.saved_tensors
        B, F = ctx.BF
        gy = grad_y.to(x2.dtype).contiguous().view(x2.shape)
        grad_x = layer.stack_backward(ctx.cfg, x2, g, saved, gy, B, F)
        return grad_x.view(ctx.shape), None, None


class LIFStack(torch.nn.Module):
    """2 or 3 LIF layers joined by fixed per-feature gains (gains: [L-1, F], the feature axis
    last), run as one fused kernel per direction: the same spikes as LIFLayer followed by
    GainLIF layers, without their intermediate tensors."""

    def __init__(self, gains: torch.Tensor, decay: float, v_th: float, v_reset: float = 0.0, alpha: float = 4.0,
                 reset: str = "hard"):
        super().__init__()
        self.register_buffer("gains", gains.detach().to(torch.float32).contiguous())
        self.decay, self.v_th, self.v_reset, self.alpha, self.reset = decay, v_th, v_reset, alpha, reset

    def cfg(self, dtype: torch.dtype) -> layer.LifConfig:
        return layer.LifConfig(self.decay, self.v_th, self.v_reset, self.alpha, self.reset, _IO[dtype], "io")

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        return FusedLIFStack.apply(x, self.gains, self.cfg(x.dtype))

    def extra_repr(self) -> str:
        return (f"layers={self.gains.shape[0] + 1}, features={self.gains.shape[1]}, decay={self.decay}, "
                f"v_th={self.v_th}, v_reset={self.v_reset}, alpha={self.alpha}, reset={self.reset}")
