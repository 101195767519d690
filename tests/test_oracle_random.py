"""Randomised pins of the CPU oracle over its hyper-parameters: decay in [0, 1], threshold,
reset value, surrogate sharpness and reset mode drawn by hypothesis (derandomised, so every
run draws the same cases) instead of the fixed sets the pins in oracle_pins.py use.

* the surrogate backward equals the gradient of the smooth model (central finite
  differences in fp64, as in pin_fd_backward);
* the fp32 forward agrees with an fp64 run of Eq. (1)-(2) within a forward-error bound
  derived from the number of roundings per step, and fires identically until the fp64
  membrane first comes within that bound of the threshold;
* splitting the sequence at any step and handing over (v, y) forward and dL/dv backward
  reproduces the single run bit for bit (Sec. 3.2);
* finite differences through 2- and 3-layer stacks joined by random gains confirm the
  oracle's stack backward for every layer.

CPU only."""
import numpy as np
import pytest
from hypothesis import HealthCheck, assume, given, settings
from hypothesis import strategies as st

import oracle
from tests import oracle_pins as P

EPS32 = 2.0 ** -24


def _f32(v):
    return float(np.float32(v))


PARAMS = st.builds(
    lambda decay, th, rest, alpha, soft: oracle.Params(_f32(decay), _f32(th), _f32(rest), _f32(alpha), soft),
    st.floats(0.0, 1.0), st.floats(0.2, 2.0), st.floats(-0.5, 0.5), st.floats(1.0, 8.0), st.booleans())

SETTINGS = settings(max_examples=40, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


@SETTINGS
@given(p=PARAMS, T=st.integers(1, 6), N=st.integers(1, 3), seed=st.integers(0, 2 ** 31 - 1))
def test_fd_identity_random_params(lib, p, T, N, seed):
    rng = np.random.default_rng(seed)
    x, gy = P._fd_inputs(rng, p, T, N)
    P._fd_case(lib, p, x, gy)


@SETTINGS
@given(p=PARAMS, seed=st.integers(0, 2 ** 31 - 1))
def test_fp64_forward_random_params(lib, p, seed):
    rng = np.random.default_rng(seed)
    T, N = 24, 48
    x = rng.normal(0.6 * p.v_th, 0.4 * p.v_th + 0.1, size=(T, N)).astype(np.float32)
    v64, y64 = P._smooth_model(p, x.astype(np.float64))
    y, v = oracle.forward(p, x, lib=lib)
    # Each step rounds at most three times (soft: v - V_th, k w, + x; hard: k v, + x) values
    # bounded by the running maximum M of |v|, |x|, |V_rest| and V_th, and |k| <= 1 carries
    # earlier errors without growth: |v - v64| <= 3 (t + 1) 2^-24 M_t (doubled for margin).
    scale = np.maximum.accumulate(np.abs(v64) + np.abs(x) + abs(p.v_rest) + abs(p.v_th), axis=0)
    bound = 6.0 * np.arange(1, T + 1)[:, None] * EPS32 * scale
    assert np.all(np.abs(v.astype(np.float64) - v64) <= bound)
    near = np.abs(v64 - p.v_th) <= bound
    ok = ~(np.cumsum(near, axis=0) > 0)
    assert np.array_equal(y[ok], y64.astype(np.uint8)[ok])


@SETTINGS
@given(p=PARAMS, T=st.integers(2, 20), split=st.integers(1, 19), seed=st.integers(0, 2 ** 31 - 1))
def test_temporal_split_random(lib, p, T, split, seed):
    a = 1 + (split - 1) % (T - 1)   # a split point strictly inside [1, T)
    rng = np.random.default_rng(seed)
    x = rng.normal(0.6 * p.v_th, 0.5 * p.v_th + 0.1, size=(T, 9)).astype(np.float32)
    gy = rng.normal(size=(T, 9))
    y, v = oracle.forward(p, x, lib=lib)
    g = oracle.backward(p, v, y, gy, lib=lib).g
    y1, v1 = oracle.forward(p, x[:a], lib=lib)
    y2, v2 = oracle.forward(p, x[a:], v_init=v1[-1], y_init=y1[-1], lib=lib)
    assert np.array_equal(np.vstack([y1, y2]), y) and np.array_equal(np.vstack([v1, v2]), v)
    g2 = oracle.backward(p, v2, y2, gy[a:], lib=lib).g
    g1 = oracle.backward(p, v1, y1, gy[:a], g_next=g2[0], lib=lib).g
    assert np.array_equal(np.vstack([g1, g2]), g)


@SETTINGS
@given(p=PARAMS, L=st.integers(2, 3), T=st.integers(1, 5), B=st.integers(1, 2), F=st.integers(1, 3),
       seed=st.integers(0, 2 ** 31 - 1))
def test_fd_stack_random_params(lib, p, L, T, B, F, seed):
    """Finite differences through a stack of L layers joined by random per-feature gains
    (either sign) confirm every layer's dL/dx of the oracle's stack, as pin_fd_stack does for
    fixed hyper-parameters."""
    rng = np.random.default_rng(seed)
    for _ in range(40):   # inputs whose fp64 trajectories stay clear of V_th in every layer
        x = rng.normal(p.v_th * 0.7, abs(p.v_th) * 0.6 + 0.2, size=(T, B * F)).astype(np.float32)
        gains = [rng.uniform(-0.8, 2.2, size=F).astype(np.float32) for _ in range(L - 1)]
        if all(np.all(np.abs(v - p.v_th) > 2e-3) for v, _ in P._smooth_stack(p, x, gains, B)):
            break
    else:
        assume(False)
    P._stack_fd_case(lib, p, x, gains, B, F, rng.normal(size=(T, B * F)))
