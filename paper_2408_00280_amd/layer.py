"""Torch-tensor conveniences over the C ABI: allocate outputs with torch, call the kernels.

Torch provides device memory and streams only; the LIF arithmetic runs in the HIP
kernels reached through :mod:`paper_2408_00280_amd.native`.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import native

IO_DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16}


@dataclass(frozen=True)
class LifConfig:
    """Hyper-parameters of one LIF layer (see snn_lif_cfg in include/snn_lif.h)."""
    decay: float
    v_th: float
    v_reset: float = 0.0
    alpha: float = 4.0
    reset: str = "hard"   # "hard" (Eq. (1)) or "soft"
    io: str = "f32"       # dtype of x, dL/dy, dL/dx
    spk: str = "u8"       # "u8", "bits", or "io" (0/1 in the I/O dtype, shaped like x)

    def c(self) -> native.snn_lif_cfg:
        return native.make_cfg(self.decay, self.v_th, self.v_reset, self.alpha, self.reset, self.io, self.spk)

    @property
    def dtype(self) -> torch.dtype:
        return IO_DTYPES[self.io]


def _require(ok: bool, what: str):
    if not ok:
        raise ValueError(what)


def _TN(x: torch.Tensor):
    T = x.shape[0]
    return T, (x.numel() // T if T else 0)


def alloc_forward(cfg: LifConfig, T: int, N: int, device, v_out: bool = False):
    """(spikes, saved uint8 bytes, v [T][N] float32 or None).  Spikes are [T][row_bytes]
    uint8 for "u8"/"bits" and [T][N] of the I/O dtype for "io"."""
    c = cfg.c()
    row = native.snn_spike_row_bytes(c, N)
    if cfg.spk == "io":
        spikes = torch.empty((T, N), dtype=cfg.dtype, device=device)
    else:
        spikes = torch.empty((T, row), dtype=torch.uint8, device=device)
    saved = torch.empty(native.snn_lif_saved_bytes(c, T, N), dtype=torch.uint8, device=device)
    v = torch.empty((T, N), dtype=torch.float32, device=device) if v_out else None
    return spikes, saved, v


def forward(cfg: LifConfig, x: torch.Tensor, *, v_out: bool = False, out=None, v_in=None, v_last=None,
            stream=None):
    """Fused forward of x[T, ...] (cfg.dtype, contiguous).  Returns (spikes, saved, v_or_None).
    v_in / v_last ([N] float32): segment state of a sequence split along time."""
    _require(x.dtype == cfg.dtype and x.is_contiguous(), f"x must be a contiguous {cfg.dtype} tensor")
    T, N = _TN(x)
    spikes, saved, v = out if out is not None else alloc_forward(cfg, T, N, x.device, v_out)
    sv = saved if saved.numel() else None
    if v_in is None and v_last is None:
        native.snn_lif_forward(cfg.c(), T, N, x, spikes, sv, v, stream)
    else:
        native.snn_lif_forward_seg(cfg.c(), T, N, x, v_in, spikes, sv, v_last, v, stream)
    return spikes, saved, v


def backward(cfg: LifConfig, x: torch.Tensor, saved: torch.Tensor, grad_s: torch.Tensor, *,
             grad_x: torch.Tensor | None = None, v_in=None, g_in=None, g_out=None, stream=None) -> torch.Tensor:
    """Fused backward; returns dL/dx with x's shape and dtype (in place if grad_x is grad_s).
    v_in / g_in / g_out ([N] float32): segment state of a sequence split along time."""
    _require(grad_s.dtype == cfg.dtype and grad_s.shape == x.shape and grad_s.is_contiguous(),
             f"grad_s must be a contiguous {cfg.dtype} tensor shaped like x")
    T, N = _TN(x)
    if grad_x is None:
        grad_x = torch.empty_like(grad_s)
    sv = saved if saved.numel() else None
    if v_in is None and g_in is None and g_out is None:
        native.snn_lif_backward(cfg.c(), T, N, x, sv, grad_s, grad_x, stream)
    else:
        native.snn_lif_backward_seg(cfg.c(), T, N, x, v_in, sv, grad_s, g_in, grad_x, g_out, stream)
    return grad_x


def _check_gain_inputs(cfg: LifConfig, spikes_in: torch.Tensor, gain: torch.Tensor, T: int, B: int, F: int):
    N = B * F
    if cfg.spk == "io":
        _require(spikes_in.dtype == cfg.dtype and tuple(spikes_in.shape) == (T, N),
                 f"spikes_in must be a {cfg.dtype} tensor of shape ({T}, {N})")
    else:
        row = native.snn_spike_row_bytes(cfg.c(), N)
        _require(spikes_in.dtype == torch.uint8 and tuple(spikes_in.shape) == (T, row),
                 f"spikes_in must be a uint8 tensor of shape ({T}, {row})")
    _require(spikes_in.is_contiguous(), "spikes_in must be contiguous")
    _require(gain.dtype == torch.float32 and gain.numel() == F and gain.is_contiguous(),
             f"gain must be a contiguous float32 tensor of {F} values")


def forward_gain(cfg: LifConfig, spikes_in: torch.Tensor, gain: torch.Tensor, B: int, F: int, *,
                 v_out: bool = False, out=None, stream=None):
    """Forward of the layer fed gain[f] * spikes_in (the previous layer's spikes, this cfg's
    u8/bits format, [T][row_bytes]).  Returns (spikes, saved, v_or_None)."""
    T = spikes_in.shape[0]
    N = B * F
    _check_gain_inputs(cfg, spikes_in, gain, T, B, F)
    spikes, saved, v = out if out is not None else alloc_forward(cfg, T, N, spikes_in.device, v_out)
    native.snn_lif_forward_gain(cfg.c(), T, B, F, spikes_in, gain, spikes, saved if saved.numel() else None, v,
                                stream)
    return spikes, saved, v


def backward_gain(cfg: LifConfig, spikes_in: torch.Tensor, gain: torch.Tensor, saved: torch.Tensor,
                  grad_s: torch.Tensor, B: int, F: int, *, grad_s_in: torch.Tensor | None = None,
                  stream=None) -> torch.Tensor:
    """Backward of forward_gain; returns dL/d spikes_in = gain[f] * dL/dx, [T][N] in cfg's I/O
    dtype (in place if grad_s_in is grad_s)."""
    T = spikes_in.shape[0]
    _check_gain_inputs(cfg, spikes_in, gain, T, B, F)
    _require(grad_s.dtype == cfg.dtype and tuple(grad_s.shape) == (T, B * F) and grad_s.is_contiguous(),
             f"grad_s must be a contiguous {cfg.dtype} tensor of shape ({T}, {B * F})")
    if grad_s_in is None:
        grad_s_in = torch.empty_like(grad_s)
    native.snn_lif_backward_gain(cfg.c(), T, B, F, spikes_in, gain, saved if saved.numel() else None, grad_s,
                                 grad_s_in, stream)
    return grad_s_in


def stack_forward(cfg: LifConfig, x: torch.Tensor, gains: torch.Tensor, B: int, F: int, *, hidden: bool = False,
                  v_out: bool = False, stream=None):
    """Forward of len(gains) + 1 layers fused across depth (gains: float32 [L-1, F]) on
    x[T, ...] (cfg.dtype, N = B*F per step).  Returns (spikes of the last layer, hidden
    spikes [L-1, T, ...] or None, saved, membranes [L, T, N] or None)."""
    _require(x.dtype == cfg.dtype and x.is_contiguous(), f"x must be a contiguous {cfg.dtype} tensor")
    _require(gains.dtype == torch.float32 and gains.dim() == 2 and gains.shape[1] == F and gains.is_contiguous(),
             f"gains must be a contiguous float32 tensor of shape (L-1, {F})")
    T, N = _TN(x)
    _require(N == B * F, "x must hold B*F neurons per step")
    L = gains.shape[0] + 1
    c = cfg.c()
    row = native.snn_spike_row_bytes(c, N)
    shape = (T, N) if cfg.spk == "io" else (T, row)
    sdt = cfg.dtype if cfg.spk == "io" else torch.uint8
    spikes = torch.empty(shape, dtype=sdt, device=x.device)
    hid = torch.empty((L - 1, *shape), dtype=sdt, device=x.device) if hidden else None
    saved = torch.empty(native.snn_lif_stack_saved_bytes(c, L, T, N), dtype=torch.uint8, device=x.device)
    v = torch.empty((L, T, N), dtype=torch.float32, device=x.device) if v_out else None
    native.snn_lif_stack_forward(c, L, T, B, F, x, gains, spikes, hid, saved if saved.numel() else None, v, stream)
    return spikes, hid, saved, v


def stack_backward(cfg: LifConfig, x: torch.Tensor, gains: torch.Tensor, saved: torch.Tensor, grad_s: torch.Tensor,
                   B: int, F: int, *, grad_x: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Backward of stack_forward: dL/dx of layer 0 from dL/dy of the last layer."""
    _require(grad_s.dtype == cfg.dtype and grad_s.shape == x.shape and grad_s.is_contiguous(),
             f"grad_s must be a contiguous {cfg.dtype} tensor shaped like x")
    T, N = _TN(x)
    L = gains.shape[0] + 1
    if grad_x is None:
        grad_x = torch.empty_like(grad_s)
    native.snn_lif_stack_backward(cfg.c(), L, T, B, F, x, gains, saved if saved.numel() else None, grad_s, grad_x,
                                  stream)
    return grad_x
