"""Launch geometry, determinism and error behaviour on the GPU.

* Neurons are independent (Sec. 3.1), so a layer cut into column slices -- which the
  library runs with other lane widths, chunk plans and grids -- must give, neuron for
  neuron, the same spikes, membranes and gradients as the whole layer, bit for bit.
* Repeated runs of the same layer are bitwise identical.
* A call rejected with an error status writes nothing."""
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


def _run(H, cfg, x, gs):
    spikes, saved, v = H.layer.forward(cfg, x, v_out=True)
    gx = H.layer.backward(cfg, x, saved, gs)
    return spikes, v, gx


def _spikes01(H, spikes, N, spk):
    """Spikes as a [T][N] 0/1 uint8 device tensor, whatever the format."""
    torch = H.torch
    if spk == "u8":
        return spikes[:, :N]
    if spk == "io":
        return (spikes != 0).to(torch.uint8)
    n = torch.arange(N, device=spikes.device)
    return ((spikes[:, n >> 3].to(torch.int32) >> (n & 7).to(torch.int32)) & 1).to(torch.uint8)


# (T, N, io, spk, reset, cut points): the whole layer and its slices fall on different plans
GEOMETRY = [
    (40, 1 << 21, "bf16", "bits", "hard", [1 << 19, (1 << 21) - 3]),   # 8/4 lanes | 2 lanes, double-buffered | 1 lane
    (40, 1 << 21, "f32", "u8", "soft", [1 << 19, (1 << 21) - 1]),       # 2 lanes | 2 lanes, double-buffered | 1 lane, 32-step chunks | 1 lane, double-buffered
    (24, 3 << 19, "bf16", "io", "soft", [4096, 3 << 18]),                # 4 lanes | 2 lanes | 2 lanes
    (9, 1 << 20, "f32", "bits", "hard", [7, 1 << 19]),                   # 16-step single chunk at 1 and 2 lanes
]


@pytest.mark.parametrize("T,N,io,spk,reset,cuts", GEOMETRY, ids=lambda v: str(v))
def test_neuron_slices_match_whole_layer(H, T, N, io, spk, reset, cuts):
    torch = H.torch
    w = H.W.custom(f"geo{T}x{N}", T, N, H.W.LifParams(0.5, 1.0, reset=reset), seed=T + N, io=io, spk=spk,
                   x_dist=("normal", 0.5, 0.5))
    cfg = H.cfg_of(w)
    x, gs = H.upload_rows(w, "x"), H.upload_rows(w, "gs")
    spikes, v, gx = _run(H, cfg, x, gs)
    y = _spikes01(H, spikes, N, spk)
    bounds = [0] + cuts + [N]
    for a, b in zip(bounds[:-1], bounds[1:]):
        xs, gss = x[:, a:b].contiguous(), gs[:, a:b].contiguous()
        s2, v2, g2 = _run(H, cfg, xs, gss)
        assert torch.equal(_spikes01(H, s2, b - a, spk), y[:, a:b]), f"spikes of neurons [{a}, {b})"
        assert torch.equal(v2.view(torch.int32), v[:, a:b].contiguous().view(torch.int32)), f"membranes [{a}, {b})"
        assert torch.equal(g2.view(torch.uint8), gx[:, a:b].contiguous().view(torch.uint8)), f"dL/dx [{a}, {b})"
    torch.cuda.synchronize()
    del x, gs, spikes, v, gx
    torch.cuda.empty_cache()


@pytest.mark.parametrize("wl", ["long", "stack", "large_T16"])
def test_ten_runs_bitwise_identical(H, wl):
    torch = H.torch
    w = H.W.WORKLOADS["large"].with_T(16) if wl == "large_T16" else H.W.WORKLOADS[wl]
    cfg = H.cfg_of(w)
    x, gs = H.upload_rows(w, "x"), H.upload_rows(w, "gs")
    first = [t.clone() for t in _run(H, cfg, x, gs)]
    for _ in range(9):
        again = _run(H, cfg, x, gs)
        for a, b in zip(again, first):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8))
    torch.cuda.synchronize()
    del x, gs, first
    torch.cuda.empty_cache()


def test_rejected_calls_write_nothing(H):
    torch = H.torch
    nat = H.native
    T, N = 40, 4096
    good = H.layer.LifConfig(0.5, 1.0)
    bad = H.layer.LifConfig(1.5, 1.0)                    # decay outside [0, 1]
    x = torch.ones((T, N), device=H.DEV)
    spikes, saved, v = H.layer.alloc_forward(good, T, N, H.DEV, v_out=True)
    gx = torch.empty((T, N), device=H.DEV)
    outs = [spikes, saved, v, gx]
    for t in outs:
        t.view(torch.uint8).fill_(0xC3)
    calls = [
        lambda: nat.snn_lif_forward(bad.c(), T, N, x, spikes, saved, v),
        lambda: nat.snn_lif_forward(good.c(), T, N, x.data_ptr() + 4, spikes, saved, v),       # misaligned
        lambda: nat.snn_lif_forward(good.c(), T, N, x, spikes, None, v),                        # saved missing
        lambda: nat.snn_lif_backward(bad.c(), T, N, x, saved, x, gx),
        lambda: nat.snn_lif_backward(good.c(), T, N, x, saved, x, gx.data_ptr() + 8),           # misaligned
        lambda: nat.snn_lif_forward_seg(good.c(), T, N, x, v.data_ptr() + 4, spikes, saved, v[0]),
        lambda: nat.snn_lif_forward_gain(good.c(), T, 2, N // 2, spikes.data_ptr() + 1, x[0], spikes, saved),
    ]
    for call in calls:
        with pytest.raises(nat.SnnError):
            call()
    torch.cuda.synchronize()
    for t in outs:
        assert bool((t.view(torch.uint8) == 0xC3).all()), "a rejected call wrote output"
    assert np.isfinite(x.cpu().numpy()).all()
