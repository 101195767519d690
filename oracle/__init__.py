"""CPU oracle for the temporally fused LIF layer -- TEST INFRASTRUCTURE ONLY.

Python marshalling over the plain C reference in ``lif_oracle.c`` (see
``lif_oracle.h`` for what it computes, its precision and its pins).  Only the
tests, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline`` leg may
import this package; the product path (``paper_2408_00280_amd``) never does.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lif_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c11", "-fPIC", "-shared"]
_lib = None


def build(src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile the oracle (always recompiles).  `src`/`out` let tests build variants."""
    subprocess.run(["gcc", *CFLAGS, "-I", _HERE, src, "-o", out + ".tmp", "-lm"], check=True)
    os.replace(out + ".tmp", out)
    return out


class _Params(ctypes.Structure):
    _fields_ = [("decay", ctypes.c_float), ("v_th", ctypes.c_float), ("v_rest", ctypes.c_float),
                ("alpha", ctypes.c_float), ("soft_reset", ctypes.c_int)]


def load(path: str = _LIB_PATH):
    """Load a built oracle library (the default one is built on first use)."""
    global _lib
    if path == _LIB_PATH and _lib is not None:
        return _lib
    if not os.path.exists(path):
        if path != _LIB_PATH:
            raise FileNotFoundError(path)
        build()
    lib = ctypes.CDLL(path)
    P, i64, vp = ctypes.POINTER(_Params), ctypes.c_int64, ctypes.c_void_p
    lib.lif_oracle_forward.argtypes = [P, i64, i64, vp, vp, vp, vp, vp]
    lib.lif_oracle_backward.argtypes = [P, i64, i64, vp, vp, vp, vp, vp, vp, vp]
    lib.lif_oracle_gain_forward.argtypes = [i64, i64, i64, vp, vp, vp]
    lib.lif_oracle_gain_backward.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp]
    for f in ("lif_oracle_forward", "lif_oracle_backward", "lif_oracle_gain_forward",
              "lif_oracle_gain_backward"):
        getattr(lib, f).restype = None
    if path == _LIB_PATH:
        _lib = lib
    return lib


@dataclass(frozen=True)
class Params:
    decay: float
    v_th: float
    v_rest: float = 0.0
    alpha: float = 4.0
    soft_reset: bool = False

    @staticmethod
    def of(p) -> "Params":
        """From any object with decay/v_th/v_reset/alpha/reset attributes (a workload's)."""
        return Params(float(p.decay), float(p.v_th), float(getattr(p, "v_reset", 0.0)),
                      float(p.alpha), getattr(p, "reset", "hard") == "soft")

    def _c(self):
        return _Params(self.decay, self.v_th, self.v_rest, self.alpha, int(self.soft_reset))


def _c32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _c64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a):
    return None if a is None else a.ctypes.data


def forward(p: Params, x, v_init=None, y_init=None, lib=None):
    """Eqs. (1)-(2) over x[T][N] (float32).  Returns (y uint8 [T][N], v float32 [T][N])."""
    lib = lib or load()
    x = _c32(x)
    T, N = x.shape
    y = np.empty((T, N), dtype=np.uint8)
    v = np.empty((T, N), dtype=np.float32)
    vi = None if v_init is None else _c32(v_init)
    yi = None if y_init is None else np.ascontiguousarray(y_init, dtype=np.uint8)
    pc = p._c()
    lib.lif_oracle_forward(ctypes.byref(pc), T, N, _ptr(x), _ptr(vi), _ptr(yi), _ptr(y), _ptr(v))
    return y, v


def backward(p: Params, v, y, gy, gy_mag=None, g_next=None, lib=None):
    """Eq. (3) in reverse time, fp64.  Returns (gx float64 [T][N], bound float64 [T][N])."""
    lib = lib or load()
    v = _c32(v)
    T, N = v.shape
    y = np.ascontiguousarray(y, dtype=np.uint8)
    gy = _c64(gy)
    gy_mag = np.abs(gy) if gy_mag is None else _c64(gy_mag)
    gn = None if g_next is None else _c64(g_next)
    assert y.shape == v.shape == gy.shape == gy_mag.shape
    gx = np.empty((T, N), dtype=np.float64)
    gm = np.empty((T, N), dtype=np.float64)
    pc = p._c()
    lib.lif_oracle_backward(ctypes.byref(pc), T, N, _ptr(v), _ptr(y), _ptr(gy), _ptr(gy_mag),
                            _ptr(gn), _ptr(gx), _ptr(gm))
    return gx, gm


def gain_forward(y, gain, B: int, F: int, lib=None):
    """x_next[t][b][f] = gain[f] * y[t][b][f]; y is uint8 [T][B*F]."""
    lib = lib or load()
    y = np.ascontiguousarray(y, dtype=np.uint8)
    T = y.shape[0]
    assert y.size == T * B * F
    g = _c32(gain)
    out = np.empty((T, B * F), dtype=np.float32)
    lib.lif_oracle_gain_forward(T, B, F, _ptr(y), _ptr(g), _ptr(out))
    return out


def gain_backward(gx_next, gx_next_mag, gain, B: int, F: int, lib=None):
    """gy[t][b][f] = gain[f] * gx_next[t][b][f] (fp64) and its bound."""
    lib = lib or load()
    gx_next = _c64(gx_next)
    gx_next_mag = _c64(gx_next_mag)
    T = gx_next.shape[0]
    g = _c32(gain)
    gy = np.empty((T, B * F), dtype=np.float64)
    gm = np.empty((T, B * F), dtype=np.float64)
    lib.lif_oracle_gain_backward(T, B, F, _ptr(gx_next), _ptr(gx_next_mag), _ptr(g), _ptr(gy), _ptr(gm))
    return gy, gm


def stack_forward(p: Params, x1, gains, B: int, F: int, lib=None):
    """L stacked layers, layer l+1 fed gains[l][f] * spikes of layer l.
    Returns per-layer lists (xs, ys, vs)."""
    xs, ys, vs = [_c32(x1)], [], []
    for l in range(len(gains) + 1):
        y, v = forward(p, xs[l], lib=lib)
        ys.append(y)
        vs.append(v)
        if l < len(gains):
            xs.append(gain_forward(y, gains[l], B, F, lib=lib))
    return xs, ys, vs


def stack_backward(p: Params, ys, vs, gy_last, gains, B: int, F: int, lib=None):
    """Backward through the stack.  Returns per-layer lists (gxs, bounds), layer 0 first."""
    L = len(ys)
    gxs, gms = [None] * L, [None] * L
    gy, gym = _c64(gy_last), np.abs(_c64(gy_last))
    for l in range(L - 1, -1, -1):
        gxs[l], gms[l] = backward(p, vs[l], ys[l], gy, gym, lib=lib)
        if l > 0:
            gy, gym = gain_backward(gxs[l], gms[l], gains[l - 1], B, F, lib=lib)
    return gxs, gms
