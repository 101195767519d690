"""The autograd binding (FusedLIF / LIFLayer) against the CPU oracle: spikes, and input
gradients from torch's autograd through one layer and through two layers joined by a
per-feature gain (a torch elementwise product standing in for an ANN operator)."""
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


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("reset", ["hard", "soft"])
def test_lif_layer_autograd(H, dtype, reset):
    torch = H.torch
    from paper_2408_00280_amd.autograd import LIFLayer
    T, shape = 21, (3, 5, 67)    # a multi-dimensional per-step shape, N = 1005 (ragged)
    N = int(np.prod(shape))
    p = H.W.LifParams(0.75, 1.0, reset=reset)
    w = H.W.custom("autograd", T, N, p, io=dtype, spk="io", seed=31, x_dist=("normal", 0.5, 0.6))
    x_np, gs_np = H.W.x_full(w), H.W.gs_full(w)
    x = H.to_dev(x_np, dtype).view(T, *shape).requires_grad_(True)
    gs = H.to_dev(gs_np, dtype).view(T, *shape)
    lif = LIFLayer(p.decay, p.v_th, p.v_reset, p.alpha, reset)
    y = lif(x)
    assert y.shape == x.shape and y.dtype == x.dtype
    (y * gs).sum().backward()
    torch.cuda.synchronize()
    P = H.oracle.Params.of(p)
    y_ref, v_ref = H.oracle.forward(P, x_np)
    ref = H.oracle.backward(P, v_ref, y_ref, gs_np)
    rep = H.parity.compare_forward(H.to_host_f32(y.detach()).reshape(T, N).astype(np.uint8), y_ref, v_ref, p.v_th)
    H.parity.compare_grad(H.to_host_f32(x.grad).reshape(T, N), ref, dtype, rep)
    assert rep.ok(), str(rep)


def test_two_layers_with_gain(H):
    """LIF -> y * gain[f] -> LIF, gradients through torch autograd vs the oracle's stack."""
    torch = H.torch
    from paper_2408_00280_amd.autograd import LIFLayer
    T, B, F = 32, 8, 256
    p = H.W.HARD_05
    w = H.W.custom("two", T, B * F, p, seed=41, spk="io", x_dist=("normal", 0.4, 0.6))
    x_np, gs_np = H.W.x_full(w), H.W.gs_full(w)
    gain_np = np.random.default_rng(5).uniform(0.5, 2.0, size=F).astype(np.float32)
    x = torch.from_numpy(x_np).to(H.DEV).view(T, B, F).requires_grad_(True)
    gain = torch.from_numpy(gain_np).to(H.DEV)
    lif = LIFLayer(p.decay, p.v_th)
    y2 = lif(lif(x) * gain)
    (y2 * torch.from_numpy(gs_np).to(H.DEV).view(T, B, F)).sum().backward()
    torch.cuda.synchronize()
    P = H.oracle.Params.of(p)
    xs, ys, vs = H.oracle.stack_forward(P, x_np, [gain_np], B, F)
    refs = H.oracle.stack_backward(P, ys, vs, gs_np, [gain_np], B, F)
    rep = H.parity.compare_forward(H.to_host_f32(y2.detach()).reshape(T, -1).astype(np.uint8), ys[1], vs[1], p.v_th)
    H.parity.compare_grad(H.to_host_f32(x.grad).reshape(T, -1), refs[0], "f32", rep)
    assert rep.ok(), str(rep)


def test_inside_sequential(H):
    """LIFLayer composes with torch modules (the paper's nn.Sequential usage)."""
    torch = H.torch
    from paper_2408_00280_amd.autograd import LIFLayer
    torch.manual_seed(0)
    model = torch.nn.Sequential(torch.nn.Linear(64, 128), LIFLayer(0.5, 1.0), torch.nn.Linear(128, 10)).to(H.DEV)
    x = torch.randn(16, 4, 64, device=H.DEV)     # [T, batch, features]
    out = model(x)
    out.sum().backward()
    assert out.shape == (16, 4, 10)
    assert all(p.grad is not None and torch.isfinite(p.grad).all() for p in model.parameters())


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fused_stack_autograd(H, dtype):
    """LIFLayer -> GainLIF(gain_12) -> GainLIF(gain_23): three layers, the later two fed
    straight from spikes; the last layer's spikes and x.grad from torch's autograd against
    the oracle's stack (the gain rounded to the I/O dtype in both directions, as the kernels
    apply it; in bf16 the gradient each layer hands down is a bf16 tensor)."""
    torch = H.torch
    from paper_2408_00280_amd.autograd import GainLIF, LIFLayer
    T, B, F = 24, 6, 1000
    p = H.W.LifParams(0.5, 1.0)
    w = H.W.custom("fstack", T, B * F, p, seed=43, io=dtype, spk="io", x_dist=("normal", 0.4, 0.6))
    x_np, gs_np = H.W.x_full(w), H.W.gs_full(w)
    rng = np.random.default_rng(7)
    gains = [rng.uniform(0.5, 2.0, size=F).astype(np.float32) for _ in range(2)]
    x = H.to_dev(x_np, dtype).view(T, B, F).requires_grad_(True)
    model = torch.nn.Sequential(LIFLayer(p.decay, p.v_th),
                                GainLIF(torch.from_numpy(gains[0]), p.decay, p.v_th),
                                GainLIF(torch.from_numpy(gains[1]), p.decay, p.v_th)).to(H.DEV)
    y = model(x)
    (y * H.to_dev(gs_np, dtype).view(T, B, F)).sum().backward()
    torch.cuda.synchronize()

    P = H.oracle.Params.of(p)
    gr = [H.round_io(g, dtype) for g in gains]
    _, ys, vs = H.oracle.stack_forward(P, x_np, gr, B, F)
    ref = H.oracle.stack_backward(P, ys, vs, gs_np, gr, B, F, rounded_handoff=dtype == "bf16")[0]
    rep = H.parity.compare_forward(H.to_host_f32(y.detach()).reshape(T, -1).astype(np.uint8), ys[2], vs[2], p.v_th)
    H.parity.compare_grad(H.to_host_f32(x.grad).reshape(T, -1), ref, dtype, rep)
    H.say(f"fused stack autograd {dtype}: {rep}")
    assert rep.ok(), str(rep)


def test_training_reduces_loss(H):
    """A small spiking network (Linear -> LIFLayer -> GainLIF -> mean over time -> Linear)
    trained with Adam on a seeded synthetic two-class problem: the loss must fall, i.e. the
    surrogate gradients through the fused kernels (and through the gain-fed layer into the
    first layer) are usable for training."""
    torch = H.torch
    from paper_2408_00280_amd.autograd import GainLIF, LIFLayer
    g = torch.Generator(device="cpu").manual_seed(0)
    T, B, D, Hd = 8, 256, 32, 128
    centers = torch.randn(2, D, generator=g)
    labels = torch.randint(0, 2, (B,), generator=g)
    x = (centers[labels] + 0.8 * torch.randn(B, D, generator=g)).to(H.DEV)
    labels = labels.to(H.DEV)
    gain = 0.5 + 1.5 * torch.rand(Hd, generator=g)
    torch.manual_seed(0)
    model = torch.nn.ModuleDict({"fc1": torch.nn.Linear(D, Hd), "lif1": LIFLayer(0.5, 1.0),
                                 "lif2": GainLIF(gain, 0.5, 1.0), "fc2": torch.nn.Linear(Hd, 2)}).to(H.DEV)
    opt = torch.optim.Adam(model.parameters(), lr=3e-3)

    def loss_fn():
        cur = model["fc1"](x).unsqueeze(0).expand(T, B, Hd).contiguous()   # constant input current
        s2 = model["lif2"](model["lif1"](cur))                             # spikes -> gain-fed layer
        return torch.nn.functional.cross_entropy(model["fc2"](s2.mean(0)), labels)

    first = loss_fn().item()
    for _ in range(40):
        opt.zero_grad()
        loss = loss_fn()
        loss.backward()
        opt.step()
    last = loss_fn().item()
    H.say(f"training: loss {first:.4f} -> {last:.4f}")
    assert model["fc1"].weight.grad is not None and torch.isfinite(model["fc1"].weight.grad).all()
    assert np.isfinite(last) and last < 0.8 * first


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_lif_stack_module(H, dtype):
    """LIFStack (the stack fused across depth) against LIFLayer -> GainLIF -> GainLIF: the
    same last-layer spikes bit for bit, and x.grad bit for bit in fp32 (within the bf16
    tolerance of the chain's own error in bf16, whose handed-down gradients are rounded)."""
    torch = H.torch
    from paper_2408_00280_amd.autograd import GainLIF, LIFLayer, LIFStack
    T, B, F = 20, 4, 777
    p = H.W.LifParams(0.5, 1.0, reset="soft")
    w = H.W.custom("lstack", T, B * F, p, seed=47, io=dtype, spk="io", x_dist=("normal", 0.5, 0.6))
    rng = np.random.default_rng(8)
    gains = torch.from_numpy(rng.uniform(0.5, 2.0, size=(2, F)).astype(np.float32))
    gs = H.to_dev(H.W.gs_full(w), dtype).view(T, B, F)
    outs = []
    for fused in (True, False):
        x = H.to_dev(H.W.x_full(w), dtype).view(T, B, F).requires_grad_(True)
        if fused:
            model = LIFStack(gains, p.decay, p.v_th, reset="soft").to(H.DEV)
        else:
            model = torch.nn.Sequential(LIFLayer(p.decay, p.v_th, reset="soft"),
                                        GainLIF(gains[0], p.decay, p.v_th, reset="soft"),
                                        GainLIF(gains[1], p.decay, p.v_th, reset="soft")).to(H.DEV)
        y = model(x)
        (y * gs).sum().backward()
        outs.append((y.detach(), x.grad))
    torch.cuda.synchronize()
    assert torch.equal(outs[0][0], outs[1][0])
    if dtype == "f32":
        assert torch.equal(outs[0][1].view(torch.int32), outs[1][1].view(torch.int32))
    else:
        a, b = H.to_host_f32(outs[0][1]), H.to_host_f32(outs[1][1])
        assert np.all(np.abs(a - b) <= 4e-2 * np.maximum(np.abs(a), np.abs(b)) + 1e-3)
