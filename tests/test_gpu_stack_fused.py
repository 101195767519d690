"""GPU parity of the gain-fed layer (snn_lif_forward_gain / snn_lif_backward_gain): a LIF
layer whose input current gain[f] * spikes_in is formed inside the kernel from the
previous layer's spikes.  Forward outputs are checked against the oracle (spikes exact,
membranes bit for bit) and against the unfused pair on the GPU (gain kernel, then the
dense layer: spikes, membranes and checkpoints bit for bit); the gradient passed to
spikes_in is checked against the oracle's gain * dL/dx within its error budgets.  Fixed
shapes at every lane/chunk plan, plus seeded random shapes, formats and hyper-parameters."""
import itertools

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


COMBOS = list(itertools.product(["hard", "soft"], ["f32", "bf16"], ["u8", "bits", "io"]))


def _pack(y: np.ndarray, spk: str) -> np.ndarray:
    """[T][N] 0/1 -> the library's spike rows (u8: as is; bits: little-endian bit order,
    rows padded to a multiple of 8 bytes)."""
    if spk == "u8":
        return np.ascontiguousarray(y, dtype=np.uint8)
    T, N = y.shape
    row = 8 * ((N + 63) // 64)
    return np.packbits(np.pad(y, ((0, 0), (0, 8 * row - N))), axis=1, bitorder="little")


def _inputs(T, B, F, io, seed, rate=0.35):
    rng = np.random.default_rng(seed)
    N = B * F
    y_in = (rng.random((T, N), dtype=np.float32) < rate).astype(np.uint8)
    gain = rng.uniform(-0.4, 1.6, size=F).astype(np.float32)
    gs = rng.normal(size=(T, N)).astype(np.float32)
    return y_in, gain, gs


def _oracle_layer(H, cfg, y_in, gain, gs, io, cols=None):
    """Oracle of the gain-fed layer on all neurons, or on columns `cols` (each column keeps
    its own feature's gain).  The gain enters rounded to the I/O dtype, in both directions, as
    the kernels apply it.  Returns (y, v, oracle.Grad of dL/d spikes_in)."""
    F = gain.size
    if cols is not None:
        y_in, gs = y_in[:, cols], gs[:, cols]
        gain = gain[cols % F]
        B, F = 1, cols.size
    else:
        B = y_in.shape[1] // F
    p = H.oracle.Params.of(cfg)
    gain = H.round_io(gain, io)
    y_ref, v_ref = H.oracle.forward(p, H.oracle.gain_forward(y_in, gain, B, F))
    return y_ref, v_ref, H.oracle.gain_backward(H.oracle.backward(p, v_ref, y_ref, gs), gain, B, F)


def _run(H, T, B, F, reset, io, spk, seed, n_sample=None, inplace=False, params=(0.5, 1.0, 0.0, 4.0)):
    torch = H.torch
    N = B * F
    decay, v_th, v_reset, alpha = params
    cfg = H.layer.LifConfig(decay, v_th, v_reset, alpha, reset=reset, io=io, spk=spk)
    y_in, gain, gs = _inputs(T, B, F, io, seed)
    gs = H.round_io(gs, io)
    s_in = (H.to_dev(y_in.astype(np.float32), io) if spk == "io"
            else torch.from_numpy(_pack(y_in, spk)).to(H.DEV))
    g_dev = torch.from_numpy(gain).to(H.DEV)
    gs_dev = H.to_dev(gs, io)

    spikes, saved, v = H.layer.forward_gain(cfg, s_in, g_dev, B, F, v_out=True)
    # the unfused pair on the same inputs
    x = torch.empty((T, N), dtype=cfg.dtype, device=H.DEV)
    H.native.snn_gain_spikes_forward(cfg.c(), T, B, F, s_in, g_dev, x)
    spikes_u, saved_u, v_u = H.layer.forward(cfg, x, v_out=True)
    assert torch.equal(spikes, spikes_u), "spikes differ from the unfused pair"
    assert torch.equal(saved, saved_u), "checkpoints differ from the unfused pair"
    assert torch.equal(v, v_u), "membranes differ from the unfused pair"
    del x, spikes_u, saved_u, v_u

    g_in = H.layer.backward_gain(cfg, s_in, g_dev, saved, gs_dev, B, F, grad_s_in=gs_dev if inplace else None)
    torch.cuda.synchronize()

    cols = None if n_sample is None else H.sample_columns(N, n_sample, seed=seed)
    y_ref, v_ref, gy_ref = _oracle_layer(H, cfg, y_in, gain, gs, io, cols)
    y_gpu = H.parity.unpack_spikes(H.to_host_f32(spikes) if spk == "io" else spikes.cpu().numpy(), N, spk)
    v_gpu, g_gpu = v.cpu().numpy(), H.to_host_f32(g_in)
    if cols is not None:
        y_gpu, v_gpu, g_gpu = y_gpu[:, cols], v_gpu[:, cols], g_gpu[:, cols]
    rep = H.parity.compare_forward(y_gpu, y_ref, v_ref, cfg.v_th, v_gpu=v_gpu)
    H.parity.compare_grad(g_gpu, gy_ref, io, rep)
    return rep, y_ref


SMALL = [(1, 1, 1), (2, 3, 1), (7, 7, 9), (17, 5, 13), (33, 10, 100), (40, 1, 4097), (64, 7, 10001),
         (100, 3, 1028)]


@pytest.mark.parametrize("T,B,F", SMALL, ids=lambda v: str(v))
@pytest.mark.parametrize("reset,io,spk", COMBOS, ids=lambda v: str(v))
def test_gain_layer_small(H, T, B, F, reset, io, spk):
    rep, y_ref = _run(H, T, B, F, reset, io, spk, seed=T * 1000 + B * 10 + F)
    assert rep.ok(), str(rep)


# (T, B, F) with N = B * F at the lane/chunk plans of the dense layer's plan tests
# (4, 2, 1 neurons per lane; bf16 8 per lane on the 2^22 layer; one or several chunks,
# double-buffered or not, short tail chunk).
PLANS = [
    (16, 256, 4096),        # N = 2^20
    (40, 4, 262145),        # N = 2^20 + 4
    (40, 1024, 4096),       # N = 2^22
    (16, 2, 262145),        # N = 524290
    (40, 2, 300001),        # N = 600002
    (40, 5, 52429),         # N = 262145
    (20, 17, 61681),        # N = 2^20 + 1
]


@pytest.mark.parametrize("T,B,F", PLANS, ids=lambda v: str(v))
@pytest.mark.parametrize("reset,io,spk", COMBOS, ids=lambda v: str(v))
def test_gain_layer_plans(H, T, B, F, reset, io, spk):
    rep, _ = _run(H, T, B, F, reset, io, spk, seed=7 * T + F, n_sample=1 << 12)
    assert rep.ok(), str(rep)
    H.torch.cuda.empty_cache()


def _random_cases():
    """Seeded random shapes (one chunk or several, a tail, 1 or 2 neurons per lane), formats
    and hyper-parameters (decay in [0, 1], threshold, reset value, surrogate sharpness)."""
    rng = np.random.default_rng(20240805)
    out = []
    for i in range(16):
        T = int(rng.integers(1, 81))
        B = int(rng.integers(1, 9))
        F = int(rng.integers(1, 5000))
        params = (float(rng.uniform(0, 1)), float(rng.uniform(0.2, 2.0)),
                  float(rng.choice([0.0, rng.uniform(-0.5, 0.5)])), float(rng.uniform(1.0, 8.0)))
        out.append((i, T, B, F, params, str(rng.choice(["hard", "soft"])), str(rng.choice(["f32", "bf16"])),
                    str(rng.choice(["u8", "bits", "io"]))))
    return out


@pytest.mark.parametrize("case", _random_cases(), ids=lambda c: f"rnd{c[0]}")
def test_gain_layer_random(H, case):
    i, T, B, F, params, reset, io, spk = case
    rep, _ = _run(H, T, B, F, reset, io, spk, seed=3000 + i, params=params)
    assert rep.ok(), f"{case}: {rep}"


def test_gain_layer_in_place(H):
    for io in ("f32", "bf16"):
        rep, _ = _run(H, 37, 6, 1000, "hard", io, "u8", seed=11, inplace=True)
        assert rep.ok(), str(rep)


def test_gain_layer_errors(H):
    torch = H.torch
    nat = H.native
    T, B, F = 4, 2, 64
    good = H.layer.LifConfig(0.5, 1.0)
    s_in = torch.zeros((T, B * F), dtype=torch.uint8, device=H.DEV)
    gain = torch.ones(F, dtype=torch.float32, device=H.DEV)
    spikes = torch.empty_like(s_in)
    gs = torch.zeros((T, B * F), dtype=torch.float32, device=H.DEV)
    with pytest.raises(nat.SnnError) as e:
        nat.snn_lif_forward_gain(H.layer.LifConfig(1.5, 1.0).c(), T, B, F, s_in, gain, spikes, None)
    assert e.value.status == -3
    with pytest.raises(nat.SnnError) as e:
        nat.snn_lif_forward_gain(good.c(), T, B, F, s_in, None, spikes, None)
    assert e.value.status == -1
    with pytest.raises(nat.SnnError) as e:
        nat.snn_lif_forward_gain(good.c(), T, B, F, s_in.data_ptr() + 1, gain, spikes, None)
    assert e.value.status == -4
    with pytest.raises(nat.SnnError) as e:
        nat.snn_lif_backward_gain(good.c(), T, B, F, s_in, gain, None, gs, gs.data_ptr() + 4)
    assert e.value.status == -4
    with pytest.raises(nat.SnnError) as e:
        nat.snn_lif_forward_gain(good.c(), T, -1, F, s_in, gain, spikes, None)
    assert e.value.status == -2
    # empty problems launch nothing and touch nothing
    nat.snn_lif_forward_gain(good.c(), 0, B, F, None, None, None, None)
    nat.snn_lif_forward_gain(good.c(), T, 0, F, None, None, None, None)
    nat.snn_lif_backward_gain(good.c(), T, B, 0, None, None, None, None, None)
    torch.cuda.synchronize()


@pytest.mark.parametrize("spk", ["u8", "bits", "io"])
def test_workload_stack_fused(H, spk):
    """The three-layer stack workload through the fused schedule: every layer's spikes and
    membranes, dL/dx of layer 0 and dL/dy of layers 0 and 1 against the oracle's stack."""
    from paper_2408_00280_amd import stack
    torch = H.torch
    w = H.W.WORKLOADS["stack"]
    B, F = w.dims
    cfg = H.cfg_of(w)
    cfg = H.layer.LifConfig(cfg.decay, cfg.v_th, cfg.v_reset, cfg.alpha, cfg.reset, cfg.io, spk)
    x_np, gs_np = H.W.x_full(w), H.W.gs_full(w)
    gains_np = [H.W.gain(w, l) for l in range(w.layers - 1)]
    gains = [torch.from_numpy(g).to(H.DEV) for g in gains_np]
    states = stack.forward(cfg, H.to_dev(x_np, w.io), gains, B, F, v_out=True, fused=True)
    grads = stack.backward(cfg, states, H.to_dev(gs_np, w.io), gains, B, F)
    torch.cuda.synchronize()
    assert all(s.x is None for s in states[1:])
    p = H.oracle.Params.of(w.params)
    xs, ys, vs = H.oracle.stack_forward(p, x_np, gains_np, B, F)
    refs = H.oracle.stack_backward(p, ys, vs, gs_np, gains_np, B, F)
    rep = H.parity.Report()
    for l in range(w.layers):
        sp = states[l].spikes
        r = H.parity.compare_forward(H.parity.unpack_spikes(H.to_host_f32(sp) if spk == "io" else sp.cpu().numpy(),
                                                            w.N, spk),
                                     ys[l], vs[l], w.params.v_th, v_gpu=states[l].v.cpu().numpy())
        H.say(f"fused stack layer {l} ({spk}): rate {ys[l].mean():.3f} {r}")
        assert r.ok(), f"layer {l}: {r}"
    H.parity.compare_grad(H.to_host_f32(grads[0]), refs[0], w.io, rep)
    for l in range(w.layers - 1):   # dL/dy of layer l = gain_l * dL/dx of layer l + 1
        gy = H.oracle.gain_backward(refs[l + 1], gains_np[l], B, F)
        H.parity.compare_grad(H.to_host_f32(grads[l + 1]), gy, w.io, rep)
    H.say(f"fused stack gradients ({spk}): {rep}")
    assert rep.ok(), str(rep)
