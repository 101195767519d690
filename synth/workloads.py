"""The synthetic LIF workloads: shapes, value distributions and layer hyper-parameters.

No LIF arithmetic lives here; this only says what to draw.  Tensors are
time-major ``[T][N]`` (row t at flat offset t*N); a multi-dimensional per-step
shape such as ``[B, C, H, W]`` is contiguous, so N is its product.

Stream numbers (the ``stream`` argument of the generator): 0 = input current x
of the first layer, 1 = upstream gradient dL/dy of the last layer, 2 = burst
mask, 3 + l = per-feature gain feeding layer l + 1 of a stack.  The seed is the
workload number.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np

import synth

STREAM_X = 0
STREAM_GS = 1
STREAM_BURST = 2
STREAM_GAIN0 = 3


@dataclass(frozen=True)
class LifParams:
    """LIF hyper-parameters: decay k_tau and V_rest of Eq. (1), V_th of Eq. (2), and
    the sigmoid-surrogate sharpness alpha of Sec. 5.2.  ``reset`` is "hard" (Eq. (1))
    or "soft" (subtract V_th, a variant the paper does not define)."""
    decay: float
    v_th: float
    v_reset: float = 0.0
    alpha: float = 4.0
    reset: str = "hard"


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    T: int
    dims: tuple                 # per-time-step shape; N = prod(dims)
    x_dist: tuple               # ("normal", mean, sd) or ("uniform", low, high)
    params: LifParams
    io: str = "f32"             # dtype of x, dL/dy, dL/dx: "f32" or "bf16"
    spk: str = "u8"             # spike storage: "u8" (one byte per neuron) or "bits"
    burst: tuple | None = None  # (p, value): i.i.d. entries of x overwritten by value
    layers: int = 1             # >1: a stack, layer l+1 fed gain_l[f] * spikes_l
    gain_dist: tuple | None = None
    gs_dist: tuple = ("normal", 0.0, 1.0)
    description: str = ""

    @property
    def N(self) -> int:
        return int(np.prod(self.dims))

    @property
    def F(self) -> int:
        """Features per sample: the last per-step dimension (the gain's length)."""
        return int(self.dims[-1])

    def with_T(self, T: int) -> "Workload":
        return replace(self, T=T)


HARD_05 = LifParams(decay=0.5, v_th=1.0)

WORKLOADS = {
    "single": Workload(
        "single", 1, 8, (65536,), ("normal", 0.6, 0.4), HARD_05,
        description="single LIF layer x[T=8, N=65536] fp32 ~ N(0.6, 0.4), decay 0.5, V_th 1, hard reset"),
    "conv": Workload(
        "conv", 2, 16, (64, 128, 32, 32), ("normal", 0.5, 0.5), HARD_05,
        description="conv-shaped LIF layer x[T=16, B=64, C=128, H=32, W=32] fp32 ~ N(0.5, 0.5), "
                    "decay 0.5, V_th 1, hard reset, u8 spikes"),
    "long": Workload(
        "long", 3, 128, (32, 4096), ("uniform", 0.0, 0.8),
        LifParams(decay=0.75, v_th=1.0, reset="soft"), burst=(0.1, 1.5),
        description="long-horizon LIF x[T=128, N=32x4096] fp32 ~ U(0, 0.8) with 10% bursts of 1.5, "
                    "decay 0.75, V_th 1, soft reset"),
    "stack": Workload(
        "stack", 4, 32, (128, 4096), ("normal", 0.4, 0.6), HARD_05, layers=3,
        gain_dist=("uniform", 0.5, 2.0),
        description="three stacked LIF layers x[T=32, B=128, N=4096] fp32 ~ N(0.4, 0.6), per-feature "
                    "gain ~ U(0.5, 2) between layers, decay 0.5, V_th 1, hard reset"),
    "large": Workload(
        "large", 5, 64, (1 << 24,), ("normal", 0.5, 0.5), HARD_05, io="bf16", spk="bits",
        description="large-scale LIF x[T, N=2^24] bf16 I/O ~ N(0.5, 0.5), fp32 membrane, decay 0.5, "
                    "V_th 1, hard reset, bit-packed spikes; T in {4, 16, 64, 256}"),
}
LARGE_T = (4, 16, 64, 256)

# A monolayer of 1,000,000 neurons with the paper's hyper-parameters (Sec. 5.1; the
# single-GPU time-step experiment of Sec. 5.3 uses such a layer without ANN operators).
# The paper gives no input distribution; N(0.2, 0.2) makes about a third of the steps fire.
WORKLOADS["paper_monolayer"] = Workload(
    "paper_monolayer", 6, 32, (1_000_000,), ("normal", 0.2, 0.2),
    LifParams(decay=0.2, v_th=0.3, v_reset=0.0, alpha=4.0),
    description="monolayer of 1,000,000 LIF neurons, k_tau 0.2, V_th 0.3, V_rest 0, alpha 4, "
                "x ~ N(0.2, 0.2), fp32, u8 spikes, hard reset")

# The paper's own hyper-parameters (Sec. 5.1): V_rest = 0, k_tau = 0.2, V_th = 0.3, alpha = 4.
PAPER_PARAMS = LifParams(decay=0.2, v_th=0.3, v_reset=0.0, alpha=4.0)


def _round_io(w: Workload, a: np.ndarray) -> np.ndarray:
    """Values exactly representable in the workload's I/O dtype, as float32."""
    if w.io == "bf16":
        return synth.bf16_bits_to_f32(synth.to_bf16_bits(a))
    return a


def x_rows(w: Workload, t0: int, t1: int) -> np.ndarray:
    """Rows [t0, t1) of the first layer's input current, float32 [t1-t0, N]."""
    N = w.N
    a = synth.fill(w.seed, STREAM_X, w.x_dist, (t1 - t0) * N, start=t0 * N)
    if w.burst is not None:
        synth.bernoulli_set(w.seed, STREAM_BURST, w.burst[0], w.burst[1], a, start=t0 * N)
    return _round_io(w, a).reshape(t1 - t0, N)


def gs_rows(w: Workload, t0: int, t1: int) -> np.ndarray:
    """Rows [t0, t1) of dL/dy for the last layer, float32 [t1-t0, N]."""
    N = w.N
    a = synth.fill(w.seed, STREAM_GS, w.gs_dist, (t1 - t0) * N, start=t0 * N)
    return _round_io(w, a).reshape(t1 - t0, N)


def x_full(w: Workload) -> np.ndarray:
    return x_rows(w, 0, w.T)


def gs_full(w: Workload) -> np.ndarray:
    return gs_rows(w, 0, w.T)


def x_cols(w: Workload, neurons: np.ndarray) -> np.ndarray:
    """All T rows of the input current at the given neuron columns, float32 [T, len]."""
    idx = synth.row_neuron_index(w.T, w.N, neurons)
    a = synth.gather(w.seed, STREAM_X, w.x_dist, idx.ravel())
    if w.burst is not None:
        synth.bernoulli_set_gather(w.seed, STREAM_BURST, w.burst[0], w.burst[1], idx.ravel(), a)
    return _round_io(w, a).reshape(idx.shape)


def gs_cols(w: Workload, neurons: np.ndarray) -> np.ndarray:
    idx = synth.row_neuron_index(w.T, w.N, neurons)
    a = synth.gather(w.seed, STREAM_GS, w.gs_dist, idx.ravel())
    return _round_io(w, a).reshape(idx.shape)


def gain(w: Workload, layer: int) -> np.ndarray:
    """float32 [F]: gain applied to layer `layer`'s spikes to form layer `layer+1`'s input."""
    assert w.layers > 1 and 0 <= layer < w.layers - 1
    return synth.fill(w.seed, STREAM_GAIN0 + layer, w.gain_dist, w.F)


def custom(name: str, T: int, N: int, params: LifParams, *, seed: int = 100, io: str = "f32",
           spk: str = "u8", x_dist=("normal", 0.5, 0.5), burst=None) -> Workload:
    """A small ad-hoc workload (test shapes: ragged N, tiny T, edge parameters)."""
    return Workload(name, seed, T, (N,), x_dist, params, io=io, spk=spk, burst=burst)
