"""The library under HIP graph capture and on concurrent streams.

It launches only on the caller's stream, allocates nothing and keeps no state between
calls, so (a) a forward+backward captured into a HIP graph must reproduce the eager
results on every replay, with other work and synchronizations between replays and the
outputs overwritten before each (single layers, stacks fused across depth and gain-fed
layers), and (b) layers launched on two streams at once must give the same bits as the
same layers run one after the other."""
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


CASES = [
    # (T, N, reset, io, spk): multi-chunk with a tail and double buffering; large bf16
    # layer with 8-neuron forward lanes; a short single-chunk layer; io-dtype spikes
    (40, 70001, "hard", "f32", "u8"),
    (20, 1 << 21, "soft", "bf16", "bits"),
    (4, 65536, "hard", "f32", "bits"),
    (33, 4096, "soft", "bf16", "io"),
    (72, 1 << 21, "hard", "f32", "u8"),       # several chunks in 1024-lane workgroups with barriers
    (80, 1 << 21, "soft", "bf16", "bits"),    # the same in bf16 (8-neuron forward lanes)
]


def _layer(H, T, N, reset, io, spk, seed):
    w = H.W.custom(f"g{T}x{N}", T, N, H.W.LifParams(0.5, 1.0, reset=reset), seed=seed, io=io, spk=spk,
                   x_dist=("normal", 0.5, 0.5))
    cfg = H.cfg_of(w)
    x, gs = H.to_dev(H.W.x_full(w), io), H.to_dev(H.W.gs_full(w), io)
    spikes, saved, v = H.layer.alloc_forward(cfg, T, N, H.DEV, v_out=True)
    gx = H.torch.empty_like(gs)
    return cfg, x, gs, (spikes, saved, v), gx


def _run(H, cfg, x, gs, out, gx):
    spikes, saved, v = out
    H.layer.forward(cfg, x, v_out=True, out=out)
    H.layer.backward(cfg, x, saved, gs, grad_x=gx)


@pytest.mark.parametrize("T,N,reset,io,spk", CASES, ids=lambda v: str(v))
def test_graph_replays_match_eager(H, T, N, reset, io, spk):
    torch = H.torch
    cfg, x, gs, out, gx = _layer(H, T, N, reset, io, spk, seed=T + N)
    _run(H, cfg, x, gs, out, gx)
    torch.cuda.synchronize()
    ref = [t.clone() for t in out if t is not None and t.numel()] + [gx.clone()]

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _run(H, cfg, x, gs, out, gx)
    for rep in range(3):
        for t in list(out) + [gx]:       # poison every output between replays (eager fills)
            if t is not None and t.numel():
                t.view(torch.uint8).fill_(0xA5)
        junk = torch.randn(1 << 20, device=H.DEV).sum()   # unrelated eager work
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [t for t in out if t is not None and t.numel()] + [gx]
        for a, b in zip(got, ref):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"replay {rep} differs from eager"
        del junk


def test_two_streams_concurrently(H):
    """Two different layers, each on its own stream, launched interleaved; the same bits as
    one after the other on the default stream."""
    torch = H.torch
    A = _layer(H, 40, 1 << 20, "hard", "f32", "u8", seed=1)
    B = _layer(H, 24, (1 << 20) + 2, "soft", "bf16", "bits", seed=2)
    refs = []
    for L in (A, B):
        _run(H, *L)
        torch.cuda.synchronize()
        refs.append([t.clone() for t in L[3] if t is not None and t.numel()] + [L[4].clone()])
        for t in list(L[3]) + [L[4]]:
            if t is not None and t.numel():
                t.view(torch.uint8).fill_(0x5A)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()   # default priority
    for _ in range(2):
        with torch.cuda.stream(s1):
            H.layer.forward(A[0], A[1], v_out=True, out=A[3])
        with torch.cuda.stream(s2):
            H.layer.forward(B[0], B[1], v_out=True, out=B[3])
        with torch.cuda.stream(s1):
            H.layer.backward(A[0], A[1], A[3][1], A[2], grad_x=A[4])
        with torch.cuda.stream(s2):
            H.layer.backward(B[0], B[1], B[3][1], B[2], grad_x=B[4])
    torch.cuda.synchronize()
    for L, ref in zip((A, B), refs):
        got = [t for t in L[3] if t is not None and t.numel()] + [L[4]]
        for a, b in zip(got, ref):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))
    assert np.isfinite(H.to_host_f32(A[4])).all()


STACK_CASES = [
    # (schedule, L, reset, io, spk): fused across depth (2 or 3 layers) and the gain-fed layer
    # of a stack fused across its gain; 40 steps = two 16-step chunks and a tail
    ("depth", 3, "hard", "f32", "u8"),
    ("depth", 2, "soft", "bf16", "bits"),
    ("gain", 2, "hard", "f32", "u8"),
    ("gain", 2, "soft", "bf16", "io"),
]


@pytest.mark.parametrize("schedule,L,reset,io,spk", STACK_CASES, ids=lambda v: str(v))
def test_graph_replays_stack(H, schedule, L, reset, io, spk):
    """The stack kernels captured into a HIP graph: every replay equals the eager run."""
    torch = H.torch
    T, B, F = 40, 6, 1000
    N = B * F
    cfg = H.layer.LifConfig(0.5, 1.0, reset=reset, io=io, spk=spk)
    gen = torch.Generator(device=H.DEV)
    gen.manual_seed(L * 100 + T)
    x = (torch.randn((T, N), device=H.DEV, generator=gen) * 0.6 + 0.5).to(cfg.dtype)
    gs = torch.randn((T, N), device=H.DEV, generator=gen).to(cfg.dtype)
    gains = (torch.rand((L - 1, F), device=H.DEV, generator=gen) * 1.5 + 0.5).contiguous()
    if schedule == "gain":
        spikes_in, _, _ = H.layer.forward(cfg, x)        # a first layer's spikes feed the gain

        def run():
            spikes, saved, _ = H.layer.forward_gain(cfg, spikes_in, gains[0], B, F)
            return [spikes, saved, H.layer.backward_gain(cfg, spikes_in, gains[0], saved, gs, B, F)]
    else:
        def run():
            spikes, _, saved, _ = H.layer.stack_forward(cfg, x, gains, B, F)
            return [spikes, saved, H.layer.stack_backward(cfg, x, gains, saved, gs, B, F)]

    ref = [t.clone() for t in run()]
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        outs = run()
    for rep in range(3):
        for t in outs:                   # poison every output between replays (eager fills)
            if t.numel():
                t.view(torch.uint8).fill_(0xA5)
        junk = torch.randn(1 << 20, device=H.DEV).sum()   # unrelated eager work
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs, ref):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"replay {rep} differs from eager"
        del junk
