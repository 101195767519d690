"""Comparison rules between the HIP path's outputs and the CPU oracle's.

Spikes: exact, except that a mismatch at (t, n) is forgiven when the oracle's
membrane sits strictly within 1e-5 of V_th there (an exact tie is never forgiven:
H(0) = 1 must hold bit for bit); a neuron with a forgiven mismatch is left out of
all later forward comparisons and of every backward comparison.  Membranes: bit
for bit.  Gradients: |gpu - ref| <= q |ref| + (1 + q) (RTOL err + u_bf16 rnd) + atol,
where `err` and `rnd` are the oracle's running error budgets (the rounding terms of
each step carried back through the true factor dv^{t+1}/dv^t, see oracle.Grad), q is
the unit roundoff of the stored result (2^-8 for bf16, 0 for fp32, whose stored value
is the computed one) and u_bf16 = 2^-8 scales the budget of bf16 copies of dL/dy made
between layers.  The recurrence runs in fp32 for both I/O dtypes, so RTOL = 1e-5 bounds
its per-operation error (about 170 ulps).  NaN must match NaN.  The plain relative rule
|gpu - ref| <= r |ref| (r = 1e-5 fp32, 2e-2 bf16) is counted too, for information: it
fails by design where the two terms of Eq. (3) cancel.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

NEAR_BAND = 1e-5
RTOL = 1e-5                  # per-operation relative error budget of the fp32 recurrence
BF16_U = 2.0 ** -8           # unit roundoff of bf16, round to nearest even
PLAIN_RTOL = {"f32": 1e-5, "bf16": 2e-2}   # the plain relative rule, reported only
ATOL = 1e-30


def unpack_spikes(raw: np.ndarray, N: int, spk: str) -> np.ndarray:
    """Spikes in the library's format -> [T][N] uint8 (0/1); checks padding and values.
    u8/bits: [T][row_bytes] uint8; io: [T][N] float32 (bf16 already widened)."""
    if spk == "io":
        a = np.asarray(raw, dtype=np.float32)
        assert a.shape[1] == N and np.all((a == 0) | (a == 1)), "io spikes must be exactly 0 or 1"
        return a.astype(np.uint8)
    raw = np.ascontiguousarray(raw, dtype=np.uint8)
    if spk == "u8":
        assert raw.shape[1] == N
        assert raw.max(initial=0) <= 1
        return raw
    assert raw.shape[1] == 8 * ((N + 63) // 64)
    bits = np.unpackbits(raw, axis=1, bitorder="little")
    assert not bits[:, N:].any(), "padding bits must be zero"
    return bits[:, :N]


def bf16_to_f32(a: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(a).view(np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass
class Report:
    ties: int = 0
    near: int = 0
    forgiven: int = 0
    hard: int = 0
    v_unequal: int = 0
    grad_bad: int = 0
    grad_checked: int = 0
    rel_fail: int = 0             # entries outside the plain relative rule (information only)
    max_grad_err: float = 0.0     # max |gpu - ref| / tolerance
    excluded: np.ndarray = field(default=None, repr=False)

    def ok(self) -> bool:
        return self.hard == 0 and self.v_unequal == 0 and self.grad_bad == 0

    def __str__(self):
        return (f"ties={self.ties} near={self.near} forgiven={self.forgiven} hard={self.hard} "
                f"v_unequal={self.v_unequal} grad_bad={self.grad_bad}/{self.grad_checked} "
                f"rel_fail={self.rel_fail} max_grad_err/tol={self.max_grad_err:.3g}")

    def counts(self) -> dict:
        return {"ties": self.ties, "near": self.near, "forgiven": self.forgiven, "hard": self.hard,
                "v_unequal": self.v_unequal, "grad_bad": self.grad_bad, "grad_checked": self.grad_checked,
                "rel_fail": self.rel_fail, "max_grad_err_over_tol": self.max_grad_err}


def compare_forward(y_gpu, y_ref, v_ref, v_th: float, v_gpu=None, rep: Report | None = None) -> Report:
    rep = rep or Report()
    y_gpu = np.asarray(y_gpu, dtype=np.uint8)
    y_ref = np.asarray(y_ref, dtype=np.uint8)
    th = np.float32(v_th)
    dist = np.abs(v_ref.astype(np.float64) - np.float64(th))
    rep.ties += int((v_ref == th).sum())
    near = (dist > 0) & (dist < NEAR_BAND)
    rep.near += int(near.sum())
    mism = y_gpu != y_ref
    forgiven = mism & near
    # after the first forgiven mismatch a neuron's later steps are not compared
    after = np.cumsum(forgiven, axis=0) > 0
    later = np.zeros_like(after)
    later[1:] = after[:-1]
    rep.forgiven += int((forgiven & ~later).sum())
    rep.hard += int((mism & ~forgiven & ~later).sum())
    excluded = after.any(axis=0)
    rep.excluded = excluded if rep.excluded is None else (rep.excluded | excluded)
    if v_gpu is not None:
        a = np.asarray(v_gpu, dtype=np.float32)
        same = (a.view(np.uint32) == v_ref.view(np.uint32)) | (np.isnan(a) & np.isnan(v_ref))
        rep.v_unequal += int((~same & ~later).sum())
    return rep


def grad_tolerance(ref, io: str, rtol: float = RTOL, atol: float = ATOL) -> np.ndarray:
    """Allowed |gpu - ref| for each entry of an oracle.Grad whose GPU value is stored in `io`."""
    q = BF16_U if io == "bf16" else 0.0
    return q * np.abs(ref.g) + (1.0 + q) * (rtol * ref.err + BF16_U * ref.rnd) + atol


def compare_grad(g_gpu, ref, io: str, rep: Report, rtol: float = RTOL, atol: float = ATOL) -> Report:
    """GPU dL/dx (stored in dtype `io`, given as float values) against an oracle.Grad."""
    assert io in PLAIN_RTOL, io
    g = np.asarray(g_gpu, dtype=np.float64)
    g_ref = ref.g
    assert g.shape == g_ref.shape, (g.shape, g_ref.shape)
    keep = np.ones(g.shape, dtype=bool)
    if rep.excluded is not None:
        keep &= ~rep.excluded[None, :]
    nan_ref, nan_gpu = np.isnan(g_ref), np.isnan(g)
    bad_nan = (nan_ref != nan_gpu) & keep
    fin = keep & ~nan_ref & ~nan_gpu
    err = np.abs(g - g_ref)
    tol = grad_tolerance(ref, io, rtol, atol)
    bad = fin & ~(err <= tol)
    rep.grad_bad += int(bad.sum() + bad_nan.sum())
    rep.grad_checked += int(keep.sum())
    rep.rel_fail += int((fin & ~(err <= PLAIN_RTOL[io] * np.abs(g_ref) + atol)).sum())
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(fin, err / tol, 0.0)
    rep.max_grad_err = max(rep.max_grad_err, float(ratio.max(initial=0.0)))
    return rep
