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
    ci = ctypes.c_int
    lib.lif_oracle_backward.argtypes = [P, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.lif_oracle_gain_forward.argtypes = [i64, i64, i64, vp, vp, vp]
    lib.lif_oracle_gain_backward.argtypes = [i64, i64, i64, vp, vp, vp, vp, vp, vp, vp]
    lib.lif_oracle_stack_forward.argtypes = [P, ci, i64, i64, i64, vp, vp, vp, vp, vp]
    lib.lif_oracle_stack_backward.argtypes = [P, ci, i64, i64, i64, vp, vp, vp, vp, ci, vp, vp, vp]
    for f in ("lif_oracle_forward", "lif_oracle_backward", "lif_oracle_gain_forward",
              "lif_oracle_gain_backward", "lif_oracle_stack_forward"):
        getattr(lib, f).restype = None
    lib.lif_oracle_stack_backward.restype = ctypes.c_int
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


@dataclass
class Grad:
    """dL/dx from the oracle's backward (fp64) with its two running error budgets:
    `err` scales with the evaluation's per-operation relative error, `rnd` with the unit
    roundoff of lower-precision copies of dL/dy that fed it (see lif_oracle.h)."""
    g: np.ndarray
    err: np.ndarray
    rnd: np.ndarray

    def sel(self, idx) -> "Grad":
        """The same index applied to all three arrays."""
        return Grad(self.g[idx], self.err[idx], self.rnd[idx])

    @staticmethod
    def exact(g) -> "Grad":
        """An input known exactly (both budgets zero)."""
        g = _c64(g)
        return Grad(g, np.zeros_like(g), np.zeros_like(g))


def backward(p: Params, v, y, gy, gy_err=None, gy_rnd=None, g_next=None, lib=None) -> Grad:
    """Eq. (3) in reverse time, fp64, with its error budgets (float64 [T][N] each).
    gy_err / gy_rnd: budgets of gy when an earlier computation produced it (None: exact)."""
    lib = lib or load()
    v = _c32(v)
    T, N = v.shape
    y = np.ascontiguousarray(y, dtype=np.uint8)
    gy = _c64(gy)
    ge = None if gy_err is None else _c64(gy_err)
    gr = None if gy_rnd is None else _c64(gy_rnd)
    gn = None if g_next is None else _c64(g_next)
    assert y.shape == v.shape == gy.shape
    assert ge is None or ge.shape == gy.shape
    assert gr is None or gr.shape == gy.shape
    assert gn is None or gn.shape == (N,)
    gx = np.empty((T, N), dtype=np.float64)
    err = np.empty((T, N), dtype=np.float64)
    rnd = np.empty((T, N), dtype=np.float64)
    pc = p._c()
    lib.lif_oracle_backward(ctypes.byref(pc), T, N, _ptr(v), _ptr(y), _ptr(gy), _ptr(ge), _ptr(gr),
                            _ptr(gn), _ptr(gx), _ptr(err), _ptr(rnd))
    return Grad(gx, err, rnd)


def gain_forward(y, gain, B: int, F: int, lib=None):
    """x_next[t][b][f] = gain[f] * y[t][b][f]; y is uint8 [T][B*F]."""
    lib = lib or load()
    y = np.ascontiguousarray(y, dtype=np.uint8)
    T = y.shape[0]
    assert y.size == T * B * F
    g = _c32(gain)
    assert g.shape == (F,)
    out = np.empty((T, B * F), dtype=np.float32)
    lib.lif_oracle_gain_forward(T, B, F, _ptr(y), _ptr(g), _ptr(out))
    return out


def gain_backward(gx_next: Grad, gain, B: int, F: int, lib=None) -> Grad:
    """gy[t][b][f] = gain[f] * gx_next[t][b][f] (fp64), budgets scaled by |gain[f]|."""
    lib = lib or load()
    a, e, r = _c64(gx_next.g), _c64(gx_next.err), _c64(gx_next.rnd)
    T = a.shape[0]
    assert a.size == T * B * F and e.shape == a.shape and r.shape == a.shape
    g = _c32(gain)
    assert g.shape == (F,)
    out = [np.empty((T, B * F), dtype=np.float64) for _ in range(3)]
    lib.lif_oracle_gain_backward(T, B, F, _ptr(a), _ptr(e), _ptr(r), _ptr(g), *(_ptr(o) for o in out))
    return Grad(*out)


def _gains(gains, L: int, F: int):
    g = _c32(np.reshape(gains, (L - 1, F)) if L > 1 else np.zeros((0, F)))
    return np.ascontiguousarray(g)


def stack_forward(p: Params, x1, gains, B: int, F: int, lib=None):
    """L = len(gains) + 1 stacked layers, layer l+1 fed gains[l][f] * spikes of layer l.
    Returns per-layer lists (xs, ys, vs), layer 0 first."""
    lib = lib or load()
    x1 = _c32(x1)
    T = x1.shape[0]
    L = len(gains) + 1
    assert x1.size == T * B * F
    g = _gains(gains, L, F)
    xs = np.empty((L, T, B * F), dtype=np.float32)
    ys = np.empty((L, T, B * F), dtype=np.uint8)
    vs = np.empty((L, T, B * F), dtype=np.float32)
    pc = p._c()
    lib.lif_oracle_stack_forward(ctypes.byref(pc), L, T, B, F, _ptr(x1), _ptr(g), _ptr(xs), _ptr(ys), _ptr(vs))
    return list(xs), list(ys), list(vs)


def stack_backward(p: Params, ys, vs, gy_last, gains, B: int, F: int, rounded_handoff: bool = False,
                   lib=None) -> list:
    """Backward through the stack from the last layer's dL/dy.  Returns a list of Grad,
    dL/dx of every layer, layer 0 first.  rounded_handoff: the gradient passed down between
    layers is stored in a lower precision (bf16 tensors between autograd layers)."""
    lib = lib or load()
    L = len(ys)
    assert len(vs) == L and len(gains) == L - 1
    y = np.ascontiguousarray(np.stack(ys), dtype=np.uint8)
    v = _c32(np.stack(vs))
    _, T, N = v.shape
    assert N == B * F
    gy = _c64(gy_last)
    assert gy.shape == (T, N)
    g = _gains(gains, L, F)
    out = [np.empty((L, T, N), dtype=np.float64) for _ in range(3)]
    pc = p._c()
    rc = lib.lif_oracle_stack_backward(ctypes.byref(pc), L, T, B, F, _ptr(v), _ptr(y), _ptr(g), _ptr(gy),
                                       int(rounded_handoff), *(_ptr(o) for o in out))
    if rc != 0:
        raise MemoryError("lif_oracle_stack_backward: out of memory")
    return [Grad(out[0][l], out[1][l], out[2][l]) for l in range(L)]
