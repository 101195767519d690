"""Pins of the CPU oracle to facts fixed by the paper and by mathematics.

Each ``pin_*`` takes an oracle library handle (``oracle.load(path)``) and raises
AssertionError when the oracle disagrees.  ``test_oracle_pins.py`` runs them on
the real oracle; ``test_oracle_mutants.py`` runs them on copies of the oracle
with planted mistakes and requires each mistake to trip at least one pin.

Expected values come from closed forms (geometric sums, exact rational arithmetic),
hand-derived fixtures under ``tests/golden/``, library routines
(``scipy.special.expit``), central finite differences of a separately written smooth
model (one layer, and stacks of layers joined by a gain), and structural invariants.
The oracle's error budgets are pinned by a separately written fp32 evaluation of
Eq. (3) whose every operation is pushed by a greedy adversary (the budget must cover
it), and by their size on the long soft-reset workload (they must stay near |dL/dx|).
"""
from __future__ import annotations

import math
import os
from fractions import Fraction

import numpy as np
from scipy.special import expit

import oracle
from synth import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


def _delta_lib(alpha, u):
    """Derivative of sigmoid(alpha*u) via the library logistic: alpha s(au) s(-au)."""
    u = np.asarray(u, dtype=np.float64)
    return alpha * expit(alpha * u) * expit(-alpha * u)


def _const(T, N, c):
    return np.full((T, N), c, dtype=np.float32)


# ---------------------------------------------------------------- forward pins

def pin_constant_input_period_hard(lib):
    """Constant input, hard reset, V_rest = 0: spikes every m steps, m from the
    geometric-sum closed form in tests/golden/constant_input_periods.txt."""
    T = 40
    for c, k, m in _rows("constant_input_periods.txt"):
        c, k, m = float(c), float(k), int(m)
        # the fixture's period must follow from the closed form in exact arithmetic
        c_, k_ = Fraction(float(np.float32(c))), Fraction(float(np.float32(k)))
        ms = [j for j in range(1, 200)
              if (c_ * j if k_ == 1 else c_ * (1 - k_ ** j) / (1 - k_)) >= 1]
        assert (ms[0] if ms else 0) == m, (c, k, m)
        y, v = oracle.forward(oracle.Params(k, 1.0), _const(T, 3, c), lib=lib)
        want = np.zeros(T, dtype=np.uint8)
        if m:
            want[m - 1::m] = 1
        for n in range(3):
            assert np.array_equal(y[:, n], want), (c, k, y[:, n], want)


def pin_constant_input_rest_nonzero(lib):
    """V_rest != 0: v^0 = V_rest, and after a spike the next step starts from V_rest + c with
    no decay of V_rest (Eq. (1) at y = 1).  Between spikes, j steps after a phase that began at
    value b, v = k^j b + c (1 - k^j)/(1 - k) (geometric sum), exact for these dyadic values."""
    k, c, rest, th, T = 0.5, 0.625, 0.25, 1.0, 12
    y, v = oracle.forward(oracle.Params(k, th, rest), _const(T, 1, c), lib=lib)
    K, C, R = Fraction(k), Fraction(c), Fraction(rest)
    base, j = K * R + C, 0          # step 1: k V_rest + c
    exp_v, exp_y = [], []
    for _ in range(T):
        val = K ** j * base + C * (1 - K ** j) / (1 - K)
        fired = val >= th
        exp_v.append(val)
        exp_y.append(int(fired))
        base, j = (R + C, 0) if fired else (base, j + 1)
    assert exp_v[:4] == [Fraction(3, 4), 1, Fraction(7, 8), Fraction(17, 16)]
    assert np.array_equal(y[:, 0], np.array(exp_y, dtype=np.uint8)), (y[:, 0], exp_y)
    assert [Fraction(float(a)) for a in v[:, 0]] == exp_v


def pin_fp32_round_half_even_trap(lib):
    """c = 0.5, k = 0.5, V_th = 1 never fires in exact arithmetic (v = 1 - 2^-t), but in fp32
    v at step 25 is fl(1 - 2^-25) = 1.0 (round half to even), which fires (H(0) = 1); the reset
    restarts the same sequence, so spikes fall at steps 25, 50, 75."""
    y, v = oracle.forward(oracle.Params(0.5, 1.0), _const(80, 2, 0.5), lib=lib)
    want = np.zeros(80, dtype=np.uint8)
    want[[24, 49, 74]] = 1
    assert np.array_equal(y[:, 0], want)
    assert v[23, 0] == np.float32(1 - 2.0 ** -24) and v[24, 0] == np.float32(1.0)


def pin_soft_reset_k1_count(lib):
    """Soft reset with k = 1 and 0 <= c <= V_th: v^t = t c - V_th n_{t-1}, so the spike count
    after t steps is floor(t c / V_th) and y^t = floor(t c/V_th) - floor((t-1) c/V_th)."""
    T = 64
    for c in (0.375, 0.3125, 0.625, 1.0):
        y, _ = oracle.forward(oracle.Params(1.0, 1.0, soft_reset=True), _const(T, 2, c), lib=lib)
        t = np.arange(1, T + 1)
        want = (np.floor(t * c) - np.floor((t - 1) * c)).astype(np.uint8)
        assert np.array_equal(y[:, 0], want), c
        assert int(y[:, 1].sum()) == math.floor(T * c)


def pin_soft_reset_closed_forms(lib):
    """Soft reset, k < 1.  (i) An impulse a >= V_th then silence: one spike, after which the
    residual a - V_th leaks geometrically, v^t = k^{t-1} (a - V_th).  (ii) A constant c >= V_th
    that fires every step: v^t = v* + (c - v*) k^{t-1}, v* = (c - k V_th)/(1 - k).  With
    k = 1/2, V_th = 1, c = 3/2 that is v^t = 2 - 2^-t (reset then leak; subtracting V_th after
    the leak instead would give 1.25 at step 2)."""
    T, k = 16, 0.5
    x = np.zeros((T, 1), dtype=np.float32)
    x[0, 0] = 1.5
    y, v = oracle.forward(oracle.Params(k, 1.0, soft_reset=True), x, lib=lib)
    assert y[:, 0].tolist() == [1] + [0] * (T - 1)
    assert v[:, 0].tolist() == [1.5] + [0.5 * k ** (t - 1) for t in range(2, T + 1)]
    y, v = oracle.forward(oracle.Params(k, 1.0, soft_reset=True), _const(T, 1, 1.5), lib=lib)
    assert y[:, 0].tolist() == [1] * T
    assert v[:, 0].tolist() == [2 - 2.0 ** -t for t in range(1, T + 1)]


def pin_subthreshold_geometric_leak(lib):
    """No spike: v^t = k^t V_rest + sum_{s<=t} k^{t-s} x^s; dyadic inputs make it exact in fp32."""
    rng = np.random.default_rng(7)
    T, N, k = 12, 16, 0.5
    x = (rng.integers(-32, 33, size=(T, N)) / 256.0).astype(np.float32)   # |x| <= 1/8
    y, v = oracle.forward(oracle.Params(k, 1.0), x, lib=lib)
    assert not y.any()
    for n in range(N):
        acc = Fraction(0)
        for t in range(T):
            acc = acc * Fraction(k) + Fraction(float(x[t, n]))
            assert Fraction(float(v[t, n])) == acc
    # an impulse a at step 1 leaves a k^{t-1}
    xi = np.zeros((T, 1), dtype=np.float32)
    xi[0, 0] = 0.75
    _, v = oracle.forward(oracle.Params(0.75, 1.0), xi, lib=lib)
    assert v[:, 0].tolist() == [0.75 * 0.75 ** (t - 1) for t in range(1, T + 1)]


def pin_T1_heaviside(lib):
    """T = 1: y = H(x - V_th) with H(0) = 1, and dL/dx = dL/dy * delta(x - V_th)."""
    th, alpha = 0.3, 4.0
    x = np.array([[th - 0.5, np.nextafter(np.float32(th), np.float32(0)), th,
                   np.nextafter(np.float32(th), np.float32(1)), th + 0.5, 3.0, -2.0]], dtype=np.float32)
    y, v = oracle.forward(oracle.Params(0.2, th, alpha=alpha), x, lib=lib)
    assert y[0].tolist() == [0, 0, 1, 1, 1, 1, 0]
    assert np.array_equal(v, x)
    gy = np.array([[1.0, -2.0, 1.0, 0.5, 1.0, 3.0, 1.0]])
    gx = oracle.backward(oracle.Params(0.2, th, alpha=alpha), v, y, gy, lib=lib).g
    want = gy * _delta_lib(alpha, x.astype(np.float64) - np.float64(np.float32(th)))
    assert np.allclose(gx, want, rtol=1e-12, atol=0)
    assert abs(gx[0, 2] - alpha / 4) < 1e-15      # delta(0) = alpha / 4


def pin_decay_zero_memoryless(lib):
    """k = 0, hard reset, V_rest = 0: v^t = x^t, y^t = H(x^t - V_th), dL/dx = dL/dy delta."""
    rng = np.random.default_rng(3)
    x = rng.normal(0.5, 0.8, size=(9, 33)).astype(np.float32)
    gy = rng.normal(size=(9, 33))
    p = oracle.Params(0.0, 1.0)
    y, v = oracle.forward(p, x, lib=lib)
    assert np.array_equal(v, x) and np.array_equal(y, (x >= 1.0).astype(np.uint8))
    gx = oracle.backward(p, v, y, gy, lib=lib).g
    assert np.allclose(gx, gy * _delta_lib(4.0, x.astype(np.float64) - 1.0), rtol=1e-12, atol=1e-300)


def pin_worked_T2(lib):
    """The hand-derived T = 2 examples of tests/golden/worked_T2.txt."""
    p = oracle.Params(0.5, 1.0)
    for row in _rows("worked_T2.txt"):
        x = np.array([[float(row[1])], [float(row[2])]], dtype=np.float32)
        y, v = oracle.forward(p, x, lib=lib)
        assert v[:, 0].tolist() == [float(row[3]), float(row[4])], row
        assert y[:, 0].tolist() == [int(row[5]), int(row[6])], row
        gx = oracle.backward(p, v, y, np.ones((2, 1)), lib=lib).g
        assert abs(gx[0, 0] - float(row[7])) < 1e-9 and abs(gx[1, 0] - float(row[8])) < 1e-9, (row, gx)


# --------------------------------------------------------------- backward pins

def _smooth_model(p: oracle.Params, x, y_star=None, v_star=None):
    """fp64 forward of a smooth stand-in for the LIF layer.

    With y_star/v_star None it runs the hard model (Eq. (1) in its arithmetic form, Eq. (2))
    and returns (v, y).  Otherwise the spike is replaced by
    yhat^t = y*^t + sigmoid(alpha (v^t - V_th)) - sigmoid(alpha (v*^t - V_th)),
    which equals y* on the frozen trajectory and has derivative delta(v - V_th) there;
    it returns the list of yhat rows.  The surrogate backward of the hard layer is exactly
    the gradient of sum_t gy^t yhat^t at x = x*."""
    T, N = x.shape
    k, th, rest, a = p.decay, p.v_th, p.v_rest, p.alpha
    v = np.full(N, rest, dtype=np.float64)
    yh = np.zeros(N)
    vs, ys = [], []
    for t in range(T):
        if p.soft_reset:
            v = k * (v - th * yh) + x[t]
        else:
            v = k * v * (1 - yh) + rest * yh + x[t]
        if y_star is None:
            yh = (v - th >= 0).astype(np.float64)
        else:
            yh = y_star[t] + expit(a * (v - th)) - expit(a * (v_star[t] - th))
        vs.append(v.copy())
        ys.append(yh.copy())
    if y_star is None:
        return np.array(vs), np.array(ys)
    return np.array(ys)


def _fd_case(lib, p, x, gy, h=1e-6, rtol=2e-5):
    x64 = x.astype(np.float64)
    v_star, y_star = _smooth_model(p, x64)
    y32, v32 = oracle.forward(p, x, lib=lib)
    assert np.array_equal(y32, y_star.astype(np.uint8)), "fp32 spikes differ from fp64 ones"
    r = oracle.backward(p, v32, y32, gy, lib=lib)
    gx, gm = r.g, r.err
    T, N = x.shape
    fd = np.empty((T, N))
    for t in range(T):
        for n in range(N):
            xp, xm = x64.copy(), x64.copy()
            xp[t, n] += h
            xm[t, n] -= h
            fp = np.sum(gy * _smooth_model(p, xp, y_star, v_star))
            fm = np.sum(gy * _smooth_model(p, xm, y_star, v_star))
            fd[t, n] = (fp - fm) / (2 * h)
    err = np.abs(fd - gx)
    assert np.all(err <= rtol * gm + 1e-8), (p, np.max(err / (gm + 1e-30)))
    assert np.all(np.abs(gx) <= gm * (1 + 1e-12))


def _fd_inputs(rng, p, T, N, margin=2e-3):
    """Random inputs whose fp64 trajectory stays `margin` away from V_th."""
    while True:
        x = rng.normal(p.v_th * 0.6, p.v_th * 0.6 + 0.2, size=(T, N)).astype(np.float32)
        v, _ = _smooth_model(p, x.astype(np.float64))
        if np.all(np.abs(v - p.v_th) > margin):
            return x, rng.normal(size=(T, N))


def pin_fd_backward(lib):
    """Finite differences of the smooth model confirm the whole backward recurrence
    (hard reset at V_rest = 0 and != 0, soft reset, and the paper's k=0.2, V_th=0.3)."""
    rng = np.random.default_rng(11)
    cases = [oracle.Params(0.5, 1.0), oracle.Params(0.75, 1.0, 0.25), oracle.Params(0.75, 1.0, soft_reset=True),
             oracle.Params(0.2, 0.3), oracle.Params(0.9, 0.5, -0.1, alpha=2.0, soft_reset=True)]
    for p in cases:
        for _ in range(3):
            x, gy = _fd_inputs(rng, p, 6, 3)
            _fd_case(lib, p, x, gy)


def pin_fd_subthreshold(lib):
    """The non-spiking path alone: small inputs that never fire."""
    rng = np.random.default_rng(5)
    p = oracle.Params(0.5, 1.0)
    x = rng.uniform(-0.4, 0.45, size=(8, 4)).astype(np.float32)
    _fd_case(lib, p, x, rng.normal(size=(8, 4)))


def pin_backward_linear_in_gy(lib):
    rng = np.random.default_rng(2)
    p = oracle.Params(0.5, 1.0)
    x = rng.normal(0.6, 0.5, size=(10, 20)).astype(np.float32)
    y, v = oracle.forward(p, x, lib=lib)
    g1, g2 = rng.normal(size=(10, 20)), rng.normal(size=(10, 20))
    a = oracle.backward(p, v, y, g1, lib=lib).g
    b = oracle.backward(p, v, y, g2, lib=lib).g
    c = oracle.backward(p, v, y, g1 + 2.0 * g2, lib=lib).g
    assert np.allclose(c, a + 2.0 * b, rtol=1e-12, atol=1e-12)


def pin_neuron_permutation(lib):
    """Neurons are independent (Sec. 3.1): permuting columns permutes every output."""
    rng = np.random.default_rng(9)
    p = oracle.Params(0.75, 1.0, soft_reset=True)
    x = rng.normal(0.5, 0.5, size=(7, 31)).astype(np.float32)
    gy = rng.normal(size=(7, 31))
    perm = rng.permutation(31)
    y, v = oracle.forward(p, x, lib=lib)
    yp, vp = oracle.forward(p, x[:, perm], lib=lib)
    assert np.array_equal(yp, y[:, perm]) and np.array_equal(vp, v[:, perm])
    g = oracle.backward(p, v, y, gy, lib=lib).g
    gp = oracle.backward(p, vp, yp, gy[:, perm], lib=lib).g
    assert np.array_equal(gp, g[:, perm])


def pin_temporal_split(lib):
    """Reordering does not change results (Sec. 3.2): two time segments run back to back,
    handing over (v, y) forward and dL/dv backward, equal one fused run bit for bit."""
    rng = np.random.default_rng(4)
    for p in (oracle.Params(0.5, 1.0, 0.1), oracle.Params(0.75, 1.0, soft_reset=True)):
        x = rng.normal(0.5, 0.5, size=(13, 17)).astype(np.float32)
        gy = rng.normal(size=(13, 17))
        y, v = oracle.forward(p, x, lib=lib)
        g = oracle.backward(p, v, y, gy, lib=lib).g
        a = 5
        y1, v1 = oracle.forward(p, x[:a], lib=lib)
        y2, v2 = oracle.forward(p, x[a:], v_init=v1[-1], y_init=y1[-1], lib=lib)
        assert np.array_equal(np.vstack([y1, y2]), y) and np.array_equal(np.vstack([v1, v2]), v)
        g2 = oracle.backward(p, v2, y2, gy[a:], lib=lib).g
        g1 = oracle.backward(p, v1, y1, gy[:a], g_next=g2[0], lib=lib).g
        assert np.array_equal(np.vstack([g1, g2]), g)


def pin_fp64_brute_force(lib):
    """fp64 run of the hard model vs the fp32 oracle on random inputs: spikes agree away from
    the threshold and the membranes agree to fp32 accuracy."""
    rng = np.random.default_rng(13)
    p = oracle.Params(0.5, 1.0)
    x = rng.normal(0.6, 0.4, size=(16, 64)).astype(np.float32)
    v64, y64 = _smooth_model(p, x.astype(np.float64))
    y, v = oracle.forward(p, x, lib=lib)
    near = np.abs(v64 - 1.0) < 1e-5
    first_near = np.cumsum(near, axis=0) > 0
    ok = ~first_near
    assert np.array_equal(y[ok], y64.astype(np.uint8)[ok])
    assert np.all(np.abs(v[ok] - v64[ok]) <= 1e-6 * (1 + np.abs(v64[ok])))


def pin_gain_glue(lib):
    """The per-feature gain between stacked layers and its transpose."""
    rng = np.random.default_rng(1)
    T, B, F = 3, 4, 5
    y = rng.integers(0, 2, size=(T, B * F)).astype(np.uint8)
    g = rng.uniform(0.5, 2.0, size=F).astype(np.float32)
    xn = oracle.gain_forward(y, g, B, F, lib=lib)
    assert np.array_equal(xn.reshape(T, B, F), np.where(y.reshape(T, B, F) == 1, g, np.float32(0)))
    gxn, e, r = rng.normal(size=(3, T, B * F))
    out = oracle.gain_backward(oracle.Grad(gxn, np.abs(e), np.abs(r)), g, B, F, lib=lib)
    g64 = g.astype(np.float64)
    assert np.array_equal(out.g.reshape(T, B, F), gxn.reshape(T, B, F) * g64)
    assert np.array_equal(out.err.reshape(T, B, F), np.abs(e).reshape(T, B, F) * g64)
    assert np.array_equal(out.rnd.reshape(T, B, F), np.abs(r).reshape(T, B, F) * g64)


def pin_nonfinite(lib):
    """NaN never fires (NaN - V_th >= 0 is false) and persists; +inf fires and then resets."""
    x = np.array([[np.nan, np.inf, -np.inf], [0.25, 0.25, 0.25]], dtype=np.float32)
    y, v = oracle.forward(oracle.Params(0.5, 1.0), x, lib=lib)
    assert y[:, 0].tolist() == [0, 0] and np.isnan(v[1, 0])
    assert y[:, 1].tolist() == [1, 0] and v[1, 1] == np.float32(0.25)
    assert y[:, 2].tolist() == [0, 0] and v[1, 2] == -np.inf
    # the error budgets stay finite wherever the gradient is (an infinite membrane has
    # delta = 0 and contributes nothing), in both reset modes
    x = np.full((5, 6), 0.3, dtype=np.float32)
    x[0, 0], x[1, 1], x[2, 2], x[0, 3] = np.nan, np.inf, -np.inf, np.inf
    for soft in (False, True):
        p = oracle.Params(0.5, 1.0, soft_reset=soft)
        y, v = oracle.forward(p, x, lib=lib)
        r = oracle.backward(p, v, y, np.ones((5, 6)), lib=lib)
        fin = np.isfinite(r.g)
        assert fin[:, 4:].all() and np.all(np.isfinite(r.err[fin])), (soft, r.g, r.err)


# ----------------------------------------------------------------- stack pins

def _gain_rows(gains, l, B):
    """Per-neuron gain of the input of layer l + 1 (neuron n = b F + f has feature f)."""
    return np.tile(np.asarray(gains[l], dtype=np.float64), B)


def _smooth_stack(p, x, gains, B, stars=None, pert=None):
    """fp64 stack of len(gains) + 1 layers: layer 0 fed x, layer l > 0 fed gain_{l-1}[f] times
    the spikes of layer l - 1 of the same step, all T steps of a layer before the next.
    stars None: the hard model, returns per-layer (v, y).  Otherwise every spike is the smooth
    yhat of _smooth_model around the frozen per-layer trajectories stars[l] = (v*, y*), and
    the top layer's yhat rows are returned.  pert = (l, t, n, h) adds h to layer l's input
    current at (t, n)."""
    L = len(gains) + 1
    inp = np.asarray(x, dtype=np.float64)
    outs = []
    for l in range(L):
        xl = inp.copy()
        if pert is not None and pert[0] == l:
            xl[pert[1], pert[2]] += pert[3]
        if stars is None:
            v, y = _smooth_model(p, xl)
            outs.append((v, y))
            spikes = y
        else:
            spikes = _smooth_model(p, xl, stars[l][1], stars[l][0])
        if l < L - 1:
            inp = spikes * _gain_rows(gains, l, B)[None, :]
    return outs if stars is None else spikes


def _stack_fd_case(lib, p, x, gains, B, F, gy, h=1e-6, rtol=2e-5):
    stars = _smooth_stack(p, x, gains, B)
    _, ys, vs = oracle.stack_forward(p, x, gains, B, F, lib=lib)
    for l, (v64, y64) in enumerate(stars):
        assert np.array_equal(ys[l], y64.astype(np.uint8)), f"layer {l}: fp32 spikes differ from fp64 ones"
    refs = oracle.stack_backward(p, ys, vs, gy, gains, B, F, lib=lib)
    T, N = x.shape
    for l in range(len(gains) + 1):
        fd = np.empty((T, N))
        for t in range(T):
            for n in range(N):
                fp = np.sum(gy * _smooth_stack(p, x, gains, B, stars, (l, t, n, h)))
                fm = np.sum(gy * _smooth_stack(p, x, gains, B, stars, (l, t, n, -h)))
                fd[t, n] = (fp - fm) / (2 * h)
        g, e = refs[l].g, refs[l].err
        assert np.all(np.abs(fd - g) <= rtol * e + 1e-8), (p, l, np.max(np.abs(fd - g) / (e + 1e-30)))
        assert np.all(np.abs(g) <= e * (1 + 1e-12))


def pin_fd_stack(lib):
    """Finite differences through 2- and 3-layer smooth stacks confirm the oracle's stack
    backward for every layer: the gradient handed down is gain_l[f] times dL/dx of the layer
    above, through each layer's own membranes."""
    rng = np.random.default_rng(21)
    B, F, T = 2, 2, 5
    cases = [oracle.Params(0.5, 1.0), oracle.Params(0.75, 1.0, soft_reset=True),
             oracle.Params(0.6, 0.8, 0.1, alpha=3.0)]
    for L in (2, 3):
        for p in cases:
            for _ in range(40):   # inputs whose fp64 trajectories stay clear of V_th in every layer
                x = rng.normal(p.v_th * 0.7, p.v_th * 0.6 + 0.2, size=(T, B * F)).astype(np.float32)
                gains = [rng.uniform(-0.6, 2.2, size=F).astype(np.float32) for _ in range(L - 1)]
                if all(np.all(np.abs(v - p.v_th) > 2e-3) for v, _ in _smooth_stack(p, x, gains, B)):
                    break
            else:
                raise AssertionError("no clear inputs found")
            _stack_fd_case(lib, p, x, gains, B, F, rng.normal(size=(T, B * F)))


def pin_worked_stack_T2(lib):
    """Hand-derived two-layer examples (tests/golden/worked_stack_T2.txt): spikes, membranes
    and both layers' dL/dx, including a tie in layer 0 and a reset in layer 1."""
    p = oracle.Params(0.5, 1.0)
    gain = [np.array([1.5], dtype=np.float32)]
    for row in _rows("worked_stack_T2.txt"):
        vals = [float(a) for a in row[1:]]
        x = np.array(vals[0:2], dtype=np.float32).reshape(2, 1)
        _, ys, vs = oracle.stack_forward(p, x, gain, 1, 1, lib=lib)
        assert vs[0][:, 0].tolist() == vals[2:4] and ys[0][:, 0].tolist() == vals[4:6], row
        assert vs[1][:, 0].tolist() == vals[6:8] and ys[1][:, 0].tolist() == vals[8:10], row
        refs = oracle.stack_backward(p, ys, vs, np.ones((2, 1)), gain, 1, 1, lib=lib)
        assert np.allclose(refs[1].g[:, 0], vals[10:12], atol=1e-9, rtol=0), (row, refs[1].g)
        assert np.allclose(refs[0].g[:, 0], vals[12:14], atol=1e-9, rtol=0), (row, refs[0].g)


def pin_stack_single_layer(lib):
    """A stack of one layer is the layer; the top layer of a stack is the layer on its own
    input; a zero gain cuts the layers below off (zero input current, zero gradient)."""
    rng = np.random.default_rng(6)
    p = oracle.Params(0.75, 1.0, soft_reset=True)
    T, B, F = 9, 3, 4
    x = rng.normal(0.5, 0.6, size=(T, B * F)).astype(np.float32)
    gy = rng.normal(size=(T, B * F))
    y, v = oracle.forward(p, x, lib=lib)
    _, ys, vs = oracle.stack_forward(p, x, [], B, F, lib=lib)
    assert np.array_equal(ys[0], y) and np.array_equal(vs[0], v)
    ref = oracle.backward(p, v, y, gy, lib=lib)
    one = oracle.stack_backward(p, ys, vs, gy, [], B, F, lib=lib)[0]
    assert np.array_equal(one.g, ref.g) and np.array_equal(one.err, ref.err)
    gains = [np.zeros(F, dtype=np.float32), rng.uniform(0.5, 2.0, size=F).astype(np.float32)]
    xs, ys, vs = oracle.stack_forward(p, x, gains, B, F, lib=lib)
    assert not xs[1].any()
    y2, v2 = oracle.forward(p, xs[2], lib=lib)
    assert np.array_equal(ys[2], y2) and np.array_equal(vs[2], v2)
    refs = oracle.stack_backward(p, ys, vs, gy, gains, B, F, lib=lib)
    assert np.array_equal(refs[2].g, oracle.backward(p, v2, y2, gy, lib=lib).g)
    assert not refs[0].g.any()


# ---------------------------------------------------------- error-budget pins

U32 = 2.0 ** -24
LOG2E = 1.4426950408889634


def _bf16_round(a):
    """float32 -> nearest bf16 value (ties to even), as float32."""
    b = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return b.astype(np.uint32).view(np.float32)


def _fp32_eq3(p, v, y, gy, g_ref, ulps=0):
    """Eq. (3) evaluated in fp32 (surrogate through exp2, reciprocal, fused multiply-adds), a
    second evaluation used only to exercise the oracle's error budget.  Every operation's
    result is moved by `ulps` units of 2^-24 relative; per step and neuron a greedy adversary
    takes whichever direction (all up or all down) lands further from g_ref."""
    f = np.float32
    T, N = v.shape
    th, k, rest, alpha = f(p.v_th), f(p.decay), f(p.v_rest), f(p.alpha)
    c_exp = f(-float(alpha) * LOG2E)
    kth = f(k * th)
    gy = np.asarray(gy, dtype=np.float32)
    g = np.zeros(N, dtype=np.float32)
    out = np.empty((T, N), dtype=np.float32)
    for t in range(T - 1, -1, -1):
        vt = v[t]
        cand = []
        for s in (1.0, -1.0):
            def r(a):
                return f(np.asarray(a, dtype=np.float64) * (1.0 + s * ulps * U32))
            arg = r(f(c_exp * np.abs(f(vt - th))))
            e = r(f(np.exp2(arg.astype(np.float64))))
            rc = r(f(1.0 / (f(1.0) + e).astype(np.float64)))
            d = r(f(f(alpha * e) * f(rc * rc)))
            if p.soft_reset:
                D = r(np.float64(-kth) * d + np.float64(k))
            else:
                a1 = r(np.float64(-k) * vt + np.float64(rest))
                D = r(a1.astype(np.float64) * d + np.where(vt >= th, 0.0, np.float64(k)))
            cand.append(r(gy[t].astype(np.float64) * d + f(D * g)))
        far = np.abs(cand[0] - g_ref[t]) >= np.abs(cand[1] - g_ref[t])
        g = np.where(far, cand[0], cand[1])
        out[t] = g
    return out


def pin_error_budget_covers_fp32(lib):
    """The arithmetic budget `err` bounds the error of fp32 evaluations of Eq. (3): the plain
    one and ones pushed 4 ulps per operation by an adversary stay within 8 (ulps + 1) 2^-24 err,
    over random hyper-parameters of either reset mode and membranes far from the threshold
    (where the surrogate's exponent is large).  The rounding budget `rnd` covers a bf16 copy of
    the gradient handed between two stacked layers."""
    rng = np.random.default_rng(17)
    for case in range(12):
        p = oracle.Params(float(np.float32(rng.uniform(0.0, 1.0))), float(np.float32(rng.uniform(0.2, 2.0))),
                          float(np.float32(rng.uniform(-0.5, 0.5))), float(np.float32(rng.uniform(1.0, 8.0))),
                          bool(case % 2))
        T, N = 48, 1000
        x = rng.normal(0.6 * p.v_th, 1.5 * p.v_th + 0.3, size=(T, N)).astype(np.float32)
        gy = rng.normal(size=(T, N)).astype(np.float32)
        y, v = oracle.forward(p, x, lib=lib)
        ref = oracle.backward(p, v, y, gy, lib=lib)
        for ulps in (0, 4):
            emu = _fp32_eq3(p, v, y, gy, ref.g, ulps)
            assert np.all(np.abs(emu - ref.g) <= 8 * (ulps + 1) * U32 * ref.err + 1e-30), (case, ulps)
    # two layers joined by a gain, the gradient handed down rounded to bf16 on the way
    p = oracle.Params(0.5, 1.0)
    T, B, F = 32, 4, 250
    x = rng.normal(0.6, 0.6, size=(T, B * F)).astype(np.float32)
    gains = [rng.uniform(0.5, 2.0, size=F).astype(np.float32)]
    gy = _bf16_round(rng.normal(size=(T, B * F)).astype(np.float32))
    _, ys, vs = oracle.stack_forward(p, x, gains, B, F, lib=lib)
    refs = oracle.stack_backward(p, ys, vs, gy, gains, B, F, rounded_handoff=True, lib=lib)
    g1 = _fp32_eq3(p, vs[1], ys[1], gy, refs[1].g)
    gy0 = _bf16_round(np.float32(1) * g1 * np.tile(gains[0], B)[None, :])
    g0 = _fp32_eq3(p, vs[0], ys[0], gy0, refs[0].g)
    assert np.all(np.abs(g0 - refs[0].g) <= 8 * U32 * refs[0].err + 2.0 ** -8 * refs[0].rnd + 1e-30)
    assert np.any(np.abs(g0 - refs[0].g) > 8 * U32 * refs[0].err)   # the rounding budget is needed


def pin_error_budget_tight(lib):
    """The budget stays near |dL/dx| on the long soft-reset workload (T = 128, where a budget
    that grew geometrically backwards in time would make the check vacuous at early steps):
    at every step at least 99% of the neurons have err < 1e3 |dL/dx| and the median is below 20."""
    w = W.WORKLOADS["long"]
    cols = np.arange(0, w.N, 32)
    p = oracle.Params.of(w.params)
    y, v = oracle.forward(p, W.x_cols(w, cols), lib=lib)
    ref = oracle.backward(p, v, y, W.gs_cols(w, cols), lib=lib)
    ratio = ref.err / np.maximum(np.abs(ref.g), 1e-300)
    assert np.all(np.mean(ratio < 1e3, axis=1) >= 0.99), np.mean(ratio < 1e3, axis=1).min()
    assert np.all(np.median(ratio, axis=1) < 20), np.median(ratio, axis=1).max()


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
