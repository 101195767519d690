"""The benchmark's own parity leg (bench.parity_check) on the GPU: it passes the outputs of
a correct run and flags a spike or a gradient planted wrong in the timed buffers, for a
single layer and for the stack's schedules."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def H():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_harness
    return gpu_harness


def _bench():
    import os
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    import bench
    return bench


def test_parity_leg_single_layer(H):
    bench = _bench()
    torch = H.torch
    w = H.W.WORKLOADS["single"]
    x, gs = H.to_dev(H.W.x_full(w), w.io), H.to_dev(H.W.gs_full(w), w.io)
    spikes, v, gx = H.gpu_layer(w, x, gs, v_out=False)
    st = {"spk": [spikes], "g": [gx]}
    cols = bench.sample_columns(w.N, 2048)
    res = bench.parity_check(w, st, [], "layer by layer", cols)
    assert res["ok"] and res["hard"] == 0 and res["grad_bad"] == 0, res
    n = int(cols[1500])
    good = gx[3, n].clone()
    gx[3, n] = good * 1.001 + 1e-3                       # a gradient about 0.1% off
    res = bench.parity_check(w, st, [], "layer by layer", cols)
    assert not res["ok"] and res["grad_bad"] == 1, res
    gx[3, n] = good
    spikes[5, n] ^= 1                                    # a flipped spike (u8 format)
    res = bench.parity_check(w, st, [], "layer by layer", cols)
    assert not res["ok"] and res["hard"] >= 1, res
    torch.cuda.synchronize()


@pytest.mark.parametrize("schedule", ["layer by layer", "fused across the gain", "fused across depth"])
def test_parity_leg_stack(H, schedule):
    bench = _bench()
    from paper_2408_00280_amd import stack
    w = H.W.WORKLOADS["stack"]
    B, F = w.dims
    cfg = H.cfg_of(w)
    x, gs = H.to_dev(H.W.x_full(w), w.io), H.to_dev(H.W.gs_full(w), w.io)
    gains_np = [H.W.gain(w, l) for l in range(w.layers - 1)]
    gains = [H.torch.from_numpy(g).to(H.DEV) for g in gains_np]
    if schedule == "fused across depth":
        spikes, _, saved, _, gstack = stack.forward_depth(cfg, x, gains, B, F)
        gx = stack.backward_depth(cfg, x, gstack, saved, gs, B, F)
        st = {"spk": [None, None, spikes], "g": [gx]}
    else:
        states = stack.forward(cfg, x, gains, B, F, fused=schedule != "layer by layer")
        grads = stack.backward(cfg, states, gs, gains, B, F)
        st = {"spk": [s.spikes for s in states], "g": grads}
    H.torch.cuda.synchronize()
    cols = bench.sample_columns(w.N, 2048)
    res = bench.parity_check(w, st, gains_np, schedule, cols)
    assert res["ok"], res
    st["g"][0][7, int(cols[100])] += 1.0                 # a gradient planted wrong
    res = bench.parity_check(w, st, gains_np, schedule, cols)
    assert not res["ok"] and res["grad_bad"] >= 1, res
