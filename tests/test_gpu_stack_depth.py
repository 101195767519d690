"""GPU parity of the stack fused across depth (snn_lif_stack_forward / backward): 2 or 3
layers joined by per-feature gains in one kernel per direction.  Every layer's spikes and
membranes against the oracle run layer by layer (spikes exact, membranes bit for bit; the
gain rounded to the I/O dtype as a stored input current would be), dL/dx of the first
layer within the oracle's error budgets; and, for fp32 I/O, every output bit for bit equal to the
schedule that fuses each layer with its gain (snn_lif_forward_gain / backward_gain)."""
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


def _oracle(H, p, x_np, gs_np, gains, B, F, io):
    """The oracle's stack, layer by layer, with the gains rounded to the I/O dtype as the
    kernel applies them (the gradient handed down stays in fp32 registers): per layer
    (y, v), and dL/dx of layer 0 as an oracle.Grad."""
    P = H.oracle.Params.of(p)
    gains = [H.round_io(g, io) for g in gains]
    _, ys, vs = H.oracle.stack_forward(P, x_np, gains, B, F)
    return ys, vs, H.oracle.stack_backward(P, ys, vs, gs_np, gains, B, F)[0]


def _spikes(H, t, N, spk):
    return H.parity.unpack_spikes(H.to_host_f32(t) if spk == "io" else t.cpu().numpy(), N, spk)


def _run(H, T, B, F, L, reset, io, spk, seed, n_sample=None, inplace=False, p=None):
    torch = H.torch
    from paper_2408_00280_amd import stack
    N = B * F
    x_dist = ("normal", 0.5, 0.6) if p is None else ("normal", 0.5 * p.v_th, 0.6 * abs(p.v_th) + 0.1)
    p = p or H.W.LifParams(0.5, 1.0, reset=reset)
    w = H.W.custom(f"depth{T}x{N}", T, N, p, seed=seed, io=io, spk=spk, x_dist=x_dist)
    cfg = H.cfg_of(w)
    rng = np.random.default_rng(seed)
    gains = [rng.uniform(-0.3, 1.8, size=F).astype(np.float32) for _ in range(L - 1)]
    if n_sample is None:
        x_np, gs_np = H.W.x_full(w), H.W.gs_full(w)
        x, gs = H.to_dev(x_np, io), H.to_dev(gs_np, io)
    else:
        x, gs = H.upload_rows(w, "x"), H.upload_rows(w, "gs")
    gdev = [torch.from_numpy(g).to(H.DEV) for g in gains]
    spikes, hid, saved, v, gstack = stack.forward_depth(cfg, x, gdev, B, F, hidden=True, v_out=True)
    if inplace:
        gx = H.layer.stack_backward(cfg, x, gstack, saved, gs, B, F, grad_x=gs)
    else:
        gx = stack.backward_depth(cfg, x, gstack, saved, gs, B, F)
    torch.cuda.synchronize()

    if io == "f32" and n_sample is None and not inplace:   # bit for bit against the gain-fused schedule
        states = stack.forward(cfg, x, gdev, B, F, v_out=True, fused=True)
        grads = stack.backward(cfg, states, H.to_dev(gs_np, io), gdev, B, F)
        torch.cuda.synchronize()
        assert torch.equal(spikes, states[-1].spikes)
        for l in range(L - 1):
            assert torch.equal(hid[l], states[l].spikes), f"layer {l} spikes"
        for l in range(L):
            assert torch.equal(v[l].view(torch.int32), states[l].v.view(torch.int32)), f"layer {l} membranes"
        assert torch.equal(gx.view(torch.int32), grads[0].view(torch.int32)), "dL/dx of layer 0"

    cols = None if n_sample is None else H.sample_columns(N, n_sample, seed=seed)
    if cols is None:
        ys, vs, g_ref = _oracle(H, p, x_np, gs_np, gains, B, F, io)
        take = (lambda a: a)
    else:
        xc, gc = H.W.x_cols(w, cols), H.W.gs_cols(w, cols)
        ys, vs, g_ref = _oracle(H, p, xc, gc, [g[cols % F] for g in gains], 1, cols.size, io)
        take = (lambda a: a[:, cols])
    rep = H.parity.Report()
    for l in range(L):
        y_gpu = _spikes(H, spikes if l == L - 1 else hid[l], N, spk)
        H.parity.compare_forward(take(y_gpu), ys[l], vs[l], p.v_th, v_gpu=take(v[l].cpu().numpy()), rep=rep)
    H.parity.compare_grad(take(H.to_host_f32(gx)), g_ref, io, rep)
    return rep


COMBOS = list(itertools.product([2, 3], ["hard", "soft"], ["f32", "bf16"], ["u8", "bits", "io"]))
SMALL = [(1, 1, 1), (3, 2, 5), (16, 4, 1000), (17, 3, 333), (40, 7, 1001), (64, 2, 4096)]


@pytest.mark.parametrize("T,B,F", SMALL, ids=lambda v: str(v))
@pytest.mark.parametrize("L,reset,io,spk", COMBOS, ids=lambda v: str(v))
def test_depth_stack_small(H, T, B, F, L, reset, io, spk):
    rep = _run(H, T, B, F, L, reset, io, spk, seed=T * 100 + B + F + L)
    assert rep.ok(), str(rep)


# the stack workload's shape (one neuron per lane), plus larger layers checked on sampled
# columns: 2 neurons per lane beyond 2^20 neurons (the first even size past it included), 1
# on odd layers and up to 2^20, several chunks with a tail, short single chunks
PLANS = [(32, 128, 4096, None), (40, 512, 4096, 1 << 12), (40, 3, 349525, 1 << 12), (4, 512, 4096, 1 << 12),
         (9, 1, (1 << 20) + 1, 1 << 12), (33, 256, 4096, 1 << 12), (17, 2, (1 << 19) + 1, 1 << 12)]


@pytest.mark.parametrize("T,B,F,n_sample", PLANS, ids=lambda v: str(v))
@pytest.mark.parametrize("L,reset,io,spk", [(3, "hard", "f32", "u8"), (3, "soft", "bf16", "bits"),
                                            (2, "hard", "bf16", "io"), (3, "hard", "f32", "bits")],
                         ids=lambda v: str(v))
def test_depth_stack_plans(H, T, B, F, n_sample, L, reset, io, spk):
    rep = _run(H, T, B, F, L, reset, io, spk, seed=T + B + F, n_sample=n_sample)
    H.say(f"depth stack T={T} N={B * F} L={L} {reset} {io} {spk}: {rep}")
    assert rep.ok(), str(rep)
    H.torch.cuda.empty_cache()


def test_depth_stack_in_place(H):
    for io in ("f32", "bf16"):
        rep = _run(H, 37, 5, 800, 3, "hard", io, "u8", seed=9, inplace=True)
        assert rep.ok(), str(rep)


def test_depth_stack_errors(H):
    torch = H.torch
    nat = H.native
    cfg = H.layer.LifConfig(0.5, 1.0)
    T, B, F = 40, 2, 64
    x = torch.zeros((T, B * F), device=H.DEV)
    g = torch.ones((2, F), device=H.DEV)
    sp = torch.empty((T, B * F), dtype=torch.uint8, device=H.DEV)
    for L in (1, 4):
        with pytest.raises(nat.SnnError) as e:
            nat.snn_lif_stack_forward(cfg.c(), L, T, B, F, x, g, sp, None, None)
        assert e.value.status == -5
    with pytest.raises(nat.SnnError) as e:   # 40 steps need checkpoints
        nat.snn_lif_stack_forward(cfg.c(), 3, T, B, F, x, g, sp, None, None)
    assert e.value.status == -1
    assert nat.snn_lif_stack_saved_bytes(cfg.c(), 3, T, B * F) == 2 * 3 * B * F * 4
    assert nat.snn_lif_stack_saved_bytes(cfg.c(), 2, 16, B * F) == 0
    nat.snn_lif_stack_forward(cfg.c(), 3, 0, B, F, None, None, None, None, None)
    torch.cuda.synchronize()


def _random_cases():
    rng = np.random.default_rng(20240804)
    out = []
    for i in range(16):
        T = int(rng.integers(1, 70))
        B = int(rng.integers(1, 9))
        F = int(rng.integers(1, 3000))
        L = int(rng.choice([2, 3]))
        p = (float(rng.uniform(0, 1)), float(rng.uniform(0.2, 2.0)), float(rng.choice([0.0, rng.uniform(-0.5, 0.5)])),
             float(rng.uniform(1.0, 8.0)), str(rng.choice(["hard", "soft"])))
        out.append((i, T, B, F, L, p, str(rng.choice(["f32", "bf16"])), str(rng.choice(["u8", "bits", "io"]))))
    return out


@pytest.mark.parametrize("case", _random_cases(), ids=lambda c: f"rnd{c[0]}")
def test_depth_stack_random(H, case):
    """Seeded random depth, shapes, formats and hyper-parameters, against the oracle run
    layer by layer (and, for fp32, the gain-fused schedule bit for bit)."""
    i, T, B, F, L, (decay, v_th, v_reset, alpha, reset), io, spk = case
    p = H.W.LifParams(decay, v_th, v_reset=v_reset, alpha=alpha, reset=reset)
    rep = _run(H, T, B, F, L, reset, io, spk, seed=1000 + i, p=p)
    assert rep.ok(), f"{case}: {rep}"
