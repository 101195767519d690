"""Thin ctypes binding over the C ABI in include/snn_lif.h (libsnnlif.so).

Argument marshalling only: every step of the LIF path runs in the HIP kernels under
``csrc/``.  Functions keep the C names; tensor arguments may be torch
tensors (their ``data_ptr()`` is passed) or raw device addresses (int), and
``stream`` may be a ``torch.cuda.Stream``, a raw hipStream_t (int) or None for
torch's current stream.  A non-OK status raises :class:`SnnError`.

If the shared library is missing this module raises at import time: there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch  # loads the HIP runtime the library binds to (same soname)

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsnnlif.so")

SNN_OK = 0
SNN_RESET_HARD, SNN_RESET_SOFT = 0, 1
SNN_IO_F32, SNN_IO_BF16 = 0, 1
SNN_SPK_U8, SNN_SPK_BITS, SNN_SPK_IO = 0, 1, 2

STATUS_NAMES = {0: "SNN_OK", -1: "SNN_E_NULL", -2: "SNN_E_SHAPE", -3: "SNN_E_PARAM",
                -4: "SNN_E_ALIGN", -5: "SNN_E_UNSUPPORTED", -6: "SNN_E_LAUNCH"}

# Every symbol the header declares; a test checks the library exports all of them.
EXPORTS = ("snn_spike_row_bytes", "snn_lif_saved_bytes", "snn_lif_forward", "snn_lif_backward",
           "snn_lif_forward_seg", "snn_lif_backward_seg",
           "snn_gain_spikes_forward", "snn_gain_grad_backward", "snn_lif_forward_gain",
           "snn_lif_backward_gain", "snn_lif_stack_saved_bytes", "snn_lif_stack_forward",
           "snn_lif_stack_backward", "snn_lif_serial_forward_step",
           "snn_lif_serial_backward_step", "snn_status_str")


class SnnError(RuntimeError):
    def __init__(self, fn: str, status: int, text: str):
        super().__init__(f"{fn}: {STATUS_NAMES.get(status, status)} ({text})")
        self.status = status


class snn_lif_cfg(ctypes.Structure):
    _fields_ = [("decay", ctypes.c_float), ("v_th", ctypes.c_float), ("v_reset", ctypes.c_float),
                ("alpha", ctypes.c_float), ("reset", ctypes.c_int32), ("io", ctypes.c_int32),
                ("spk", ctypes.c_int32)]


def make_cfg(decay: float, v_th: float, v_reset: float = 0.0, alpha: float = 4.0, reset="hard",
             io="f32", spk="u8") -> snn_lif_cfg:
    """Build a cfg from Python values ("hard"/"soft", "f32"/"bf16", "u8"/"bits"/"io" or the ints)."""
    r = {"hard": SNN_RESET_HARD, "soft": SNN_RESET_SOFT}.get(reset, reset)
    d = {"f32": SNN_IO_F32, "bf16": SNN_IO_BF16}.get(io, io)
    s = {"u8": SNN_SPK_U8, "bits": SNN_SPK_BITS, "io": SNN_SPK_IO}.get(spk, spk)
    return snn_lif_cfg(decay, v_th, v_reset, alpha, r, d, s)


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "(the LIF path has no non-HIP fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    C, i64, vp, st = ctypes.POINTER(snn_lif_cfg), ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    szp = ctypes.POINTER(ctypes.c_size_t)
    sig = {
        "snn_spike_row_bytes": [C, i64, szp],
        "snn_lif_saved_bytes": [C, i64, i64, szp],
        "snn_lif_forward": [C, i64, i64, vp, vp, vp, vp, vp],
        "snn_lif_backward": [C, i64, i64, vp, vp, vp, vp, vp],
        "snn_lif_forward_seg": [C, i64, i64, vp, vp, vp, vp, vp, vp, vp],
        "snn_lif_backward_seg": [C, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp],
        "snn_gain_spikes_forward": [C, i64, i64, i64, vp, vp, vp, vp],
        "snn_gain_grad_backward": [C, i64, i64, i64, vp, vp, vp, vp],
        "snn_lif_forward_gain": [C, i64, i64, i64, vp, vp, vp, vp, vp, vp],
        "snn_lif_backward_gain": [C, i64, i64, i64, vp, vp, vp, vp, vp, vp],
        "snn_lif_stack_saved_bytes": [C, ctypes.c_int32, i64, i64, szp],
        "snn_lif_stack_forward": [C, ctypes.c_int32, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp],
        "snn_lif_stack_backward": [C, ctypes.c_int32, i64, i64, i64, vp, vp, vp, vp, vp, vp],
        "snn_lif_serial_forward_step": [C, i64, vp, vp, vp, vp, vp],
        "snn_lif_serial_backward_step": [C, i64, vp, vp, vp, vp, vp, vp],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = st
    lib.snn_status_str.argtypes = [st]
    lib.snn_status_str.restype = ctypes.c_char_p
    return lib


lib = _load()


def _ptr(a):
    if a is None:
        return None
    if isinstance(a, torch.Tensor):
        if a.numel() and not a.is_contiguous():
            raise ValueError("tensor arguments must be contiguous")
        return a.data_ptr() or None
    return int(a)


def _stream(s):
    if s is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, torch.cuda.Stream):
        return s.cuda_stream
    return int(s)


def _check(fn: str, status: int):
    if status != SNN_OK:
        raise SnnError(fn, status, lib.snn_status_str(status).decode())


def snn_status_str(status: int) -> str:
    return lib.snn_status_str(status).decode()


def snn_spike_row_bytes(cfg: snn_lif_cfg, N: int) -> int:
    out = ctypes.c_size_t(0)
    _check("snn_spike_row_bytes", lib.snn_spike_row_bytes(ctypes.byref(cfg), N, ctypes.byref(out)))
    return out.value


def snn_lif_saved_bytes(cfg: snn_lif_cfg, T: int, N: int) -> int:
    out = ctypes.c_size_t(0)
    _check("snn_lif_saved_bytes", lib.snn_lif_saved_bytes(ctypes.byref(cfg), T, N, ctypes.byref(out)))
    return out.value


def snn_lif_forward(cfg, T, N, x, spikes, saved, v_out=None, stream=None):
    _check("snn_lif_forward", lib.snn_lif_forward(ctypes.byref(cfg), T, N, _ptr(x), _ptr(spikes),
                                                  _ptr(saved), _ptr(v_out), _stream(stream)))


def snn_lif_backward(cfg, T, N, x, saved, grad_s, grad_x, stream=None):
    _check("snn_lif_backward", lib.snn_lif_backward(ctypes.byref(cfg), T, N, _ptr(x), _ptr(saved),
                                                    _ptr(grad_s), _ptr(grad_x), _stream(stream)))


def snn_lif_forward_seg(cfg, T, N, x, v_in, spikes, saved, v_last=None, v_out=None, stream=None):
    _check("snn_lif_forward_seg", lib.snn_lif_forward_seg(
        ctypes.byref(cfg), T, N, _ptr(x), _ptr(v_in), _ptr(spikes), _ptr(saved), _ptr(v_last), _ptr(v_out),
        _stream(stream)))


def snn_lif_backward_seg(cfg, T, N, x, v_in, saved, grad_s, g_in, grad_x, g_out=None, stream=None):
    _check("snn_lif_backward_seg", lib.snn_lif_backward_seg(
        ctypes.byref(cfg), T, N, _ptr(x), _ptr(v_in), _ptr(saved), _ptr(grad_s), _ptr(g_in), _ptr(grad_x),
        _ptr(g_out), _stream(stream)))


def snn_gain_spikes_forward(cfg, T, B, F, spikes, gain, x_next, stream=None):
    _check("snn_gain_spikes_forward", lib.snn_gain_spikes_forward(
        ctypes.byref(cfg), T, B, F, _ptr(spikes), _ptr(gain), _ptr(x_next), _stream(stream)))


def snn_gain_grad_backward(cfg, T, B, F, grad_x_next, gain, grad_s, stream=None):
    _check("snn_gain_grad_backward", lib.snn_gain_grad_backward(
        ctypes.byref(cfg), T, B, F, _ptr(grad_x_next), _ptr(gain), _ptr(grad_s), _stream(stream)))


def snn_lif_forward_gain(cfg, T, B, F, spikes_in, gain, spikes, saved, v_out=None, stream=None):
    _check("snn_lif_forward_gain", lib.snn_lif_forward_gain(
        ctypes.byref(cfg), T, B, F, _ptr(spikes_in), _ptr(gain), _ptr(spikes), _ptr(saved), _ptr(v_out),
        _stream(stream)))


def snn_lif_backward_gain(cfg, T, B, F, spikes_in, gain, saved, grad_s, grad_s_in, stream=None):
    _check("snn_lif_backward_gain", lib.snn_lif_backward_gain(
        ctypes.byref(cfg), T, B, F, _ptr(spikes_in), _ptr(gain), _ptr(saved), _ptr(grad_s), _ptr(grad_s_in),
        _stream(stream)))


def snn_lif_stack_saved_bytes(cfg: snn_lif_cfg, L: int, T: int, N: int) -> int:
    out = ctypes.c_size_t(0)
    _check("snn_lif_stack_saved_bytes", lib.snn_lif_stack_saved_bytes(ctypes.byref(cfg), L, T, N, ctypes.byref(out)))
    return out.value


def snn_lif_stack_forward(cfg, L, T, B, F, x, gains, spikes, hidden_spikes, saved, v_out=None, stream=None):
    _check("snn_lif_stack_forward", lib.snn_lif_stack_forward(
        ctypes.byref(cfg), L, T, B, F, _ptr(x), _ptr(gains), _ptr(spikes), _ptr(hidden_spikes), _ptr(saved),
        _ptr(v_out), _stream(stream)))


def snn_lif_stack_backward(cfg, L, T, B, F, x, gains, saved, grad_s, grad_x, stream=None):
    _check("snn_lif_stack_backward", lib.snn_lif_stack_backward(
        ctypes.byref(cfg), L, T, B, F, _ptr(x), _ptr(gains), _ptr(saved), _ptr(grad_s), _ptr(grad_x),
        _stream(stream)))


def snn_lif_serial_forward_step(cfg, N, x_t, v_prev, v_t, spikes_t, stream=None):
    _check("snn_lif_serial_forward_step", lib.snn_lif_serial_forward_step(
        ctypes.byref(cfg), N, _ptr(x_t), _ptr(v_prev), _ptr(v_t), _ptr(spikes_t), _stream(stream)))


def snn_lif_serial_backward_step(cfg, N, v_t, grad_s_t, g_next, grad_x_t, g_out=None, stream=None):
    _check("snn_lif_serial_backward_step", lib.snn_lif_serial_backward_step(
        ctypes.byref(cfg), N, _ptr(v_t), _ptr(grad_s_t), _ptr(g_next), _ptr(grad_x_t), _ptr(g_out),
        _stream(stream)))
