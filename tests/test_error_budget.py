"""The gradient comparison (tests/parity.py) is neither too tight nor vacuous, on the CPU.

The tolerance comes from the oracle's running error budgets (Eq. (3) with the rounding
terms of each step carried back through the true factor dv^{t+1}/dv^t).  Here a separately
written fp32 evaluation of Eq. (3) stands in for a correct kernel, and copies of it with
planted mistakes stand in for wrong ones:

* the fp32 evaluation passes on the long soft-reset workload and on the large bf16 one
  (rounded to bf16 when stored);
* a relative error of 1e-4 planted into any 16-step window of the long workload is flagged
  in most of that window's entries, the first window included (a budget that grew
  backwards in time would let errors in the early steps through);
* a recompute that is off by one step inside the first 16-step chunk, as a wrong
  checkpoint or buffer index would produce, is flagged;
* with bf16 storage a 1% error is flagged almost everywhere.
CPU only."""
import numpy as np
import pytest

import oracle
from synth import workloads as W
from tests import oracle_pins as P
from tests import parity


@pytest.fixture(scope="module")
def long_case():
    w = W.WORKLOADS["long"]
    cols = np.arange(0, w.N, 32)
    p = oracle.Params.of(w.params)
    gs = W.gs_cols(w, cols)
    y, v = oracle.forward(p, W.x_cols(w, cols))
    ref = oracle.backward(p, v, y, gs)
    return p, v, y, gs, ref, P._fp32_eq3(p, v, y, gs, ref.g)


def test_fp32_evaluation_passes(long_case):
    p, v, y, gs, ref, emu = long_case
    rep = parity.compare_grad(emu, ref, "f32", parity.Report())
    assert rep.grad_bad == 0 and rep.max_grad_err < 0.2, str(rep)
    # the plain relative rule fails where the two terms of Eq. (3) cancel
    assert rep.rel_fail > 0


def test_fp32_evaluation_passes_bf16_large():
    w = W.WORKLOADS["large"].with_T(64)
    cols = np.arange(0, w.N, w.N // 2048)
    p = oracle.Params.of(w.params)
    gs = W.gs_cols(w, cols)
    y, v = oracle.forward(p, W.x_cols(w, cols))
    ref = oracle.backward(p, v, y, gs)
    stored = P._bf16_round(P._fp32_eq3(p, v, y, gs, ref.g))
    rep = parity.compare_grad(stored, ref, "bf16", parity.Report())
    assert rep.grad_bad == 0, str(rep)


@pytest.mark.parametrize("t0", [0, 16, 48, 112])
def test_planted_window_error_caught(long_case, t0):
    p, v, y, gs, ref, emu = long_case
    bad = emu.astype(np.float64)
    bad[t0:t0 + 16] *= 1.0 + 1e-4
    flagged = np.abs(bad - ref.g) > parity.grad_tolerance(ref, "f32")
    assert not flagged[:t0].any() and not flagged[t0 + 16:].any()
    assert flagged[t0:t0 + 16].mean() > 0.6, flagged[t0:t0 + 16].mean()


def test_first_chunk_off_by_one_caught(long_case):
    p, v, y, gs, ref, emu = long_case
    v_bad = v.copy()
    v_bad[1:16] = v[0:15]
    rep = parity.compare_grad(P._fp32_eq3(p, v_bad, y, gs, ref.g), ref, "f32", parity.Report())
    assert rep.grad_bad > 0.1 * 16 * v.shape[1], str(rep)


def test_bf16_percent_error_caught(long_case):
    p, v, y, gs, ref, emu = long_case
    bad = P._bf16_round(emu).astype(np.float64)
    bad[:16] *= 1.01
    flagged = np.abs(bad - ref.g) > parity.grad_tolerance(ref, "bf16")
    assert flagged[:16].mean() > 0.95, flagged[:16].mean()
