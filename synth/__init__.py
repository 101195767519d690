"""Seeded synthetic inputs shared by the GPU path's tests/benchmark and the CPU oracle.

This package holds no LIF arithmetic: it only draws input currents, upstream
gradients, burst masks and gains.  Every value is a pure function of
(seed, stream, flat index) (see ``gen.c``), so a neuron subset regenerated with
:func:`gather_rows` is bit-identical to the same entries of a full tensor made
with :func:`fill`.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

# distribution kinds understood by gen.c
NORMAL = 0
UNIFORM = 1


def build() -> str:
    """Compile gen.c into libsynth.so (always recompiles)."""
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11", _SRC, "-o", _LIB_PATH + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    i64, u64, dbl, ptr = ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p
    lib.synth_fill_f32.argtypes = [u64, u64, ctypes.c_int, dbl, dbl, i64, i64, ptr]
    lib.synth_gather_f32.argtypes = [u64, u64, ctypes.c_int, dbl, dbl, ptr, i64, ptr]
    lib.synth_bernoulli_set_f32.argtypes = [u64, u64, dbl, ctypes.c_float, i64, i64, ptr]
    lib.synth_bernoulli_set_gather_f32.argtypes = [u64, u64, dbl, ctypes.c_float, ptr, i64, ptr]
    lib.synth_f32_to_bf16.argtypes = [ptr, ptr, i64]
    lib.synth_bits.argtypes = [u64, u64, u64]
    lib.synth_bits.restype = u64
    for f in ("synth_fill_f32", "synth_gather_f32", "synth_bernoulli_set_f32",
              "synth_bernoulli_set_gather_f32", "synth_f32_to_bf16"):
        getattr(lib, f).restype = None
    _lib = lib
    return lib


def _dist(dist):
    kind, a, b = dist
    return {"normal": NORMAL, "uniform": UNIFORM}[kind], float(a), float(b)


def fill(seed: int, stream: int, dist, count: int, start: int = 0, out: np.ndarray | None = None) -> np.ndarray:
    """float32 values at flat indices [start, start+count) of one stream."""
    kind, a, b = _dist(dist)
    if out is None:
        out = np.empty(count, dtype=np.float32)
    assert out.dtype == np.float32 and out.flags.c_contiguous and out.size == count
    _load().synth_fill_f32(seed, stream, kind, a, b, start, count, out.ctypes.data)
    return out


def gather(seed: int, stream: int, dist, idx: np.ndarray) -> np.ndarray:
    """float32 values at arbitrary flat indices of one stream."""
    kind, a, b = _dist(dist)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.shape, dtype=np.float32)
    _load().synth_gather_f32(seed, stream, kind, a, b, idx.ctypes.data, idx.size, out.ctypes.data)
    return out


def bernoulli_set(seed: int, stream: int, p: float, value: float, out: np.ndarray, start: int = 0) -> np.ndarray:
    """In place: entries whose uniform draw is below p become `value`."""
    assert out.dtype == np.float32 and out.flags.c_contiguous
    _load().synth_bernoulli_set_f32(seed, stream, p, value, start, out.size, out.ctypes.data)
    return out


def bernoulli_set_gather(seed: int, stream: int, p: float, value: float, idx: np.ndarray, out: np.ndarray) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    assert out.dtype == np.float32 and out.flags.c_contiguous and out.size == idx.size
    _load().synth_bernoulli_set_gather_f32(seed, stream, p, value, idx.ctypes.data, idx.size, out.ctypes.data)
    return out


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest even); returns the uint16 bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    out = np.empty(a.shape, dtype=np.uint16)
    _load().synth_f32_to_bf16(a.ctypes.data, out.ctypes.data, a.size)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns to float32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def bits(seed: int, stream: int, i: int) -> int:
    return int(_load().synth_bits(seed, stream, i))


def row_neuron_index(T: int, N: int, neurons: np.ndarray) -> np.ndarray:
    """Flat [T][N] indices of the given neuron columns, shape [T, len(neurons)]."""
    neurons = np.asarray(neurons, dtype=np.int64)
    return np.arange(T, dtype=np.int64)[:, None] * N + neurons[None, :]
