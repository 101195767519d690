"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the same seeded
inputs.  Spikes must match exactly (near-threshold rule in tests/parity.py), membranes bit
for bit, gradients within the oracle's running error budgets (tests/parity.py)."""
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


# ------------------------------------------------------------------ small random shapes

SHAPES = [(1, 1), (1, 1000), (2, 3), (7, 63), (16, 64), (17, 65), (33, 1000), (40, 4097), (15, 1027),
          (100, 256 * 4 * 3 + 4), (64, 70001),
          (4, 4097), (5, 64), (8, 1000), (12, 999)]   # the short single-chunk plans (4-, 8-, 16-step)
PARAMS = {
    "k05": dict(decay=0.5, v_th=1.0),
    "paper": dict(decay=0.2, v_th=0.3),                 # Sec. 5.1 hyper-parameters
    "rest": dict(decay=0.75, v_th=1.0, v_reset=0.25, alpha=2.0),
    "k1": dict(decay=1.0, v_th=1.0),
    "k0": dict(decay=0.0, v_th=0.5),
    "neg_th": dict(decay=0.5, v_th=-0.25),              # a negative threshold
    "rest_above": dict(decay=0.9, v_th=0.5, v_reset=0.75),  # reset value above the threshold
}
COMBOS = list(itertools.product(["hard", "soft"], ["f32", "bf16"], ["u8", "bits", "io"]))


def _workload(H, T, N, pname, reset, io, spk, seed):
    pp = dict(PARAMS[pname])
    p = H.W.LifParams(reset=reset, **pp)
    mean = 0.5 * pp["v_th"] + 0.1
    return H.W.custom(f"t{T}n{N}", T, N, p, seed=seed, io=io, spk=spk,
                      x_dist=("normal", mean, 0.6 * pp["v_th"] + 0.2))


@pytest.mark.parametrize("T,N", SHAPES, ids=lambda v: str(v))
@pytest.mark.parametrize("reset,io,spk", COMBOS, ids=lambda v: str(v))
def test_random_shapes(H, T, N, reset, io, spk):
    for i, pname in enumerate(PARAMS):
        w = _workload(H, T, N, pname, reset, io, spk, seed=1000 + 7 * T + N + i)
        rep = H.check_full(w)
        H.say(f"{w.name} {pname} {reset} {io} {spk}: {rep}")
        assert rep.ok(), f"{pname}: {rep}"
        assert rep.forgiven == 0


def test_in_place_gradient(H):
    for io in ("f32", "bf16"):
        w = _workload(H, 37, 5000, "k05", "hard", io, "u8", seed=5)
        rep = H.check_full(w, inplace=True)
        assert rep.ok(), str(rep)


def test_deterministic_bitwise(H):
    torch = H.torch
    w = H.W.WORKLOADS["long"].with_T(40)
    x, gs = H.to_dev(H.W.x_full(w), w.io), H.to_dev(H.W.gs_full(w), w.io)
    outs = [H.gpu_layer(w, x, gs) for _ in range(3)]
    for s, v, g in outs[1:]:
        assert torch.equal(s, outs[0][0]) and torch.equal(v, outs[0][1]) and torch.equal(g, outs[0][2])


def test_spike_ties_and_exact_values(H):
    """Inputs on the threshold must fire (H(0) = 1); bf16 inputs make ties frequent."""
    T, N = 24, 4096
    rng = np.random.default_rng(0)
    x = rng.choice(np.array([0.5, 0.25, 0.75, 1.0, 0.125], dtype=np.float32), size=(T, N))
    gs = rng.normal(size=(T, N)).astype(np.float32)
    for io, spk, reset in COMBOS_IO_SPK_RESET():
        w = H.W.custom("ties", T, N, H.W.LifParams(0.5, 1.0, reset=reset), io=io, spk=spk)
        gs_io = H.round_io(gs, io)   # the oracle gets the values the kernel reads
        spikes, v, gx = H.gpu_layer(w, H.to_dev(x, io), H.to_dev(gs_io, io))
        rep, (y_ref, v_ref, _) = H.compare_layer(w, spikes, v, gx, x, gs_io)
        assert rep.ties > 1000 and rep.ok(), str(rep)


def COMBOS_IO_SPK_RESET():
    return [(io, spk, reset) for reset, io, spk in COMBOS]


def test_nonfinite_inputs(H):
    T, N = 5, 64
    x = np.full((T, N), 0.3, dtype=np.float32)
    x[0, 0], x[1, 1], x[2, 2], x[0, 3] = np.nan, np.inf, -np.inf, np.inf
    gs = np.ones((T, N), dtype=np.float32)
    for reset in ("hard", "soft"):
        w = H.W.custom("nonfinite", T, N, H.W.LifParams(0.5, 1.0, reset=reset))
        spikes, v, gx = H.gpu_layer(w, H.to_dev(x, "f32"), H.to_dev(gs, "f32"))
        rep, _ = H.compare_layer(w, spikes, v, gx, x, gs)
        assert rep.ok(), str(rep)


def test_denormal_leak(H):
    """An impulse leaking by 1/2 per step passes through the fp32 denormal range to zero;
    both sides must agree bit for bit all the way (denormals are not flushed)."""
    T, N = 200, 8
    x = np.zeros((T, N), dtype=np.float32)
    x[0] = 0.75
    gs = np.ones((T, N), dtype=np.float32)
    w = H.W.custom("denormal", T, N, H.W.LifParams(0.5, 1.0))
    spikes, v, gx = H.gpu_layer(w, H.to_dev(x, "f32"), H.to_dev(gs, "f32"))
    vv = v.cpu().numpy()
    assert vv[130, 0] != 0 and abs(vv[130, 0]) < np.finfo(np.float32).tiny
    rep, _ = H.compare_layer(w, spikes, v, gx, x, gs)
    assert rep.ok(), str(rep)


def test_empty_problems(H):
    torch = H.torch
    w = H.W.custom("empty", 0, 64, H.W.HARD_05)
    x = torch.empty((0, 64), device=H.DEV)
    s, saved, v = H.layer.forward(H.cfg_of(w), x, v_out=True)
    g = H.layer.backward(H.cfg_of(w), x, saved, torch.empty_like(x))
    assert s.numel() == 0 and g.numel() == 0
    x = torch.empty((8, 0), device=H.DEV)
    s, saved, v = H.layer.forward(H.cfg_of(w), x)
    assert s.shape == (8, 0)


# ------------------------------------------------------------------ the five workloads

def test_workload_single(H):
    w = H.W.WORKLOADS["single"]
    rep = H.check_full(w)
    H.say(f"single: {rep}")
    assert rep.ok(), str(rep)


def test_workload_conv_full_size(H):
    """x[T=16, 64, 128, 32, 32] on the GPU in the benchmark's launch configuration; the oracle
    checks 65536 neuron columns (both ends plus random ones) over all 16 steps."""
    w = H.W.WORKLOADS["conv"]
    rep = H.check_sampled(w, 1 << 16)
    H.say(f"conv: {rep}")
    assert rep.ok(), str(rep)


def test_workload_long(H):
    w = H.W.WORKLOADS["long"]
    rep = H.check_full(w)
    H.say(f"long: {rep}")
    assert rep.ok(), str(rep)


@pytest.mark.parametrize("T", [4, 16, 64, 256])
def test_workload_large(H, T):
    """x[T, 2^24] bf16 with bit spikes, run whole on the GPU; the oracle checks 2^16 neuron
    columns over all T (2^20 at T = 256)."""
    w = H.W.WORKLOADS["large"].with_T(T)
    rep = H.check_sampled(w, 1 << 20 if T == 256 else 1 << 16)
    H.say(f"large T={T}: {rep}")
    assert rep.ok(), str(rep)
    H.torch.cuda.empty_cache()


@pytest.mark.parametrize("T", [32, 256])
def test_workload_paper_monolayer(H, T):
    """The paper's single-GPU workload shape (Sec. 5.3): a monolayer of 1,000,000 neurons with
    its hyper-parameters (Sec. 5.1: k_tau 0.2, V_th 0.3, V_rest 0, alpha 4), the time-step
    sweep's ends; the oracle checks 2^14 neuron columns over all T."""
    w = H.W.WORKLOADS["paper_monolayer"].with_T(T)
    rep = H.check_sampled(w, 1 << 14)
    H.say(f"paper monolayer T={T}: {rep}")
    assert rep.ok(), str(rep)


def test_max_neurons(H):
    """The largest layer the ABI accepts in one row: N = 2^31 - 1 (odd, so one neuron per
    lane: a grid of 2^31 lanes), three steps (a short chunk with a tail); sampled columns
    include both ends."""
    N = (1 << 31) - 1
    w = H.W.custom("maxN", 3, N, H.W.HARD_05, seed=31, x_dist=("normal", 0.6, 0.5))
    rep = H.check_sampled(w, 1 << 12)
    H.say(f"max N: {rep}")
    assert rep.ok(), str(rep)
    H.torch.cuda.empty_cache()


def test_workload_stack(H):
    """Three layers with per-feature gains in between; every layer's spikes, membranes,
    glue output and gradient against the oracle's stack."""
    from paper_2408_00280_amd import stack
    w = H.W.WORKLOADS["stack"]
    B, F = w.dims
    cfg = H.cfg_of(w)
    x_np, gs_np = H.W.x_full(w), H.W.gs_full(w)
    gains_np = [H.W.gain(w, l) for l in range(w.layers - 1)]
    gains = [H.torch.from_numpy(g).to(H.DEV) for g in gains_np]
    states = stack.forward(cfg, H.to_dev(x_np, w.io), gains, B, F, v_out=True)
    grads = stack.backward(cfg, states, H.to_dev(gs_np, w.io), gains, B, F)
    H.torch.cuda.synchronize()
    p = H.oracle.Params.of(w.params)
    xs, ys, vs = H.oracle.stack_forward(p, x_np, gains_np, B, F)
    refs = H.oracle.stack_backward(p, ys, vs, gs_np, gains_np, B, F)
    for l in range(w.layers):
        assert np.array_equal(states[l].x.cpu().numpy(), xs[l]), f"layer {l} input"
        rep = H.parity.compare_forward(H.parity.unpack_spikes(states[l].spikes.cpu().numpy(), w.N, w.spk),
                                       ys[l], vs[l], w.params.v_th, v_gpu=states[l].v.cpu().numpy())
        H.parity.compare_grad(H.to_host_f32(grads[l]), refs[l], w.io, rep)
        H.say(f"stack layer {l}: rate {ys[l].mean():.3f} {rep}")
        assert rep.ok(), f"layer {l}: {rep}"


@pytest.mark.parametrize("io,spk", [("f32", "u8"), ("f32", "bits"), ("f32", "io"), ("bf16", "u8"),
                                    ("bf16", "bits"), ("bf16", "io")])
# Row-walking kernels (N not a multiple of the piece width, padded spike-bit rows) and the
# flat ones: several workgroups with a partial last one, features not a multiple of the
# piece width, fewer features than a piece holds.
@pytest.mark.parametrize("T,B,F", [(3, 2, 5), (9, 7, 100), (4, 3, 1024), (5, 3, 4100), (7, 5, 1000),
                                   (3, 65, 1088), (5, 40, 8), (6, 8, 2), (4, 4, 6)])
def test_gain_glue(H, io, spk, T, B, F):
    torch = H.torch
    rng = np.random.default_rng(T * 100 + B + F)
    N = B * F
    y = rng.integers(0, 2, size=(T, N)).astype(np.uint8)
    gain = rng.uniform(0.5, 2.0, size=F).astype(np.float32)
    cfg = H.layer.LifConfig(0.5, 1.0, io=io, spk=spk)
    raw = y if spk == "u8" else np.packbits(
        np.pad(y, ((0, 0), (0, 8 * ((N + 63) // 64) * 8 - N))), axis=1, bitorder="little")
    spikes = H.to_dev(y.astype(np.float32), io) if spk == "io" else torch.from_numpy(np.ascontiguousarray(raw)).to(H.DEV)
    g = torch.from_numpy(gain).to(H.DEV)
    xn = torch.empty((T, N), dtype=cfg.dtype, device=H.DEV)
    H.native.snn_gain_spikes_forward(cfg.c(), T, B, F, spikes, g, xn)
    want = H.oracle.gain_forward(y, gain, B, F)
    if io == "bf16":
        want = H.parity.bf16_to_f32(H.synth_bf16(want))
    assert np.array_equal(H.to_host_f32(xn), want)
    gxn = rng.normal(size=(T, N)).astype(np.float32)
    if io == "bf16":
        gxn = H.parity.bf16_to_f32(H.synth_bf16(gxn))
    gs = torch.empty_like(xn)
    H.native.snn_gain_grad_backward(cfg.c(), T, B, F, H.to_dev(gxn, io), g, gs)
    # the product of the (I/O-dtype) gain and dL/dx_next, rounded once to the I/O dtype
    ref = H.oracle.gain_backward(H.oracle.Grad.exact(gxn), H.round_io(gain, io), B, F).g
    u = H.parity.BF16_U if io == "bf16" else 2.0 ** -24
    assert np.all(np.abs(H.to_host_f32(gs) - ref) <= u * np.abs(ref))
    inplace = H.to_dev(gxn, io)                         # grad_s may be grad_x_next
    H.native.snn_gain_grad_backward(cfg.c(), T, B, F, inplace, g, inplace)
    assert torch.equal(inplace.view(torch.uint8), gs.view(torch.uint8))


# Shapes that reach every lane/chunk plan of the library, run in full on the GPU and checked
# on sampled neuron columns.  Backward lanes: 2 neurons (1 when N is odd), bf16 4 on short
# layers (T <= 16) of at least 2^20 neurons; the bf16 forward takes 8 per lane from 2^21.
# Chunks: 16 steps (32 at 1 per lane, and for bf16 layers not double-buffered, whose forward
# loads them 16 rows at a time), double-buffered below 2^20 lanes, a short tail chunk when
# K does not divide T, and 4/8/16-step single chunks for short layers.  Layers of several
# chunks that are not double-buffered run in 1024-lane workgroups with a barrier per chunk.
PLAN_SHAPES = [
    (16, 1 << 20),          # one chunk (fp32 2 per lane, bf16 4)
    (40, (1 << 20) + 4),    # 2 per lane, double-buffered 16-step chunks, tail
    (40, 1 << 22),          # not double-buffered: fp32 16-step, bf16 32-step chunks (forward 8 per lane)
    (40, (1 << 22) + 6),    # the same at 2 per lane with a partial last workgroup
    (40, (1 << 22) + 8),    # bf16 forward 8 per lane with a partial last workgroup
    (72, (1 << 20) + 1),    # 1 per lane, not double-buffered 32-step chunks, tail
    (16, 524290),           # 2 per lane, one chunk
    (40, 600002),           # 2 per lane, double-buffered, tail
    (40, 262145),           # 1 per lane (odd N), double-buffered 32-step chunks, tail
    (20, (1 << 20) + 1),    # 1 per lane, one chunk
    (4, 1 << 20),           # short layers: one 4-step chunk
    (3, 1 << 21),           # 4-step chunk with a tail (bf16: 8 per lane in the forward)
    (8, 524290),            # one 8-step chunk, 2 per lane
    (6, 1 << 22),           # 8-step chunk with a tail (bf16 forward: 8 per lane)
    (12, 262145),           # one 16-step chunk at 1 per lane (whose long chunk is 32 steps)
    (24, 1 << 21),          # bf16: one 32-step chunk loaded as 16 rows + a tail; fp32: 16 + tail
]


@pytest.mark.parametrize("T,N", PLAN_SHAPES, ids=lambda v: str(v))
@pytest.mark.parametrize("reset,io,spk", COMBOS, ids=lambda v: str(v))
def test_plans(H, T, N, reset, io, spk):
    w = _workload(H, T, N, "k05", reset, io, spk, seed=77 + T + N)
    rep = H.check_sampled(w, 1 << 12, v_out=True)
    assert rep.ok(), str(rep)
