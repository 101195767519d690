"""GPU tests of the segment state handoff (snn_lif_forward_seg / snn_lif_backward_seg): a
sequence split along time into consecutive segments, each handing its last membrane
forward and its first-step gradient back, must reproduce the single call over all T bit
for bit (the temporal split of a layer), and a segment started from an arbitrary state
must match the oracle started from the same state."""
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

# (T, N, segment lengths): single- and multi-chunk segments, tails, one-step segments,
# and layer sizes that reach the 4-, 2- and 1-neuron lanes and double buffering.
SPLITS = [
    (2, 1000, [1, 1]),
    (40, 4097, [17, 23]),
    (64, 20000, [1, 31, 32]),
    (100, 70001, [50, 50]),
    (40, (1 << 20) + 4, [8, 9, 23]),
    (48, 1 << 21, [16, 32]),
    (80, 1 << 21, [40, 40]),    # multi-chunk segments in 1024-lane workgroups (bf16 too)
]


def _segments_vs_whole(H, w, lens):
    torch = H.torch
    cfg = H.cfg_of(w)
    T, N = w.T, w.N
    x_np, gs_np = H.W.x_full(w), H.W.gs_full(w)
    x, gs = H.to_dev(x_np, w.io), H.to_dev(gs_np, w.io)
    spikes, saved, v = H.layer.forward(cfg, x, v_out=True)
    gx = H.layer.backward(cfg, x, saved, gs)

    bounds = np.cumsum([0] + lens)
    assert bounds[-1] == T
    states = []
    v_in = None
    for a, b in zip(bounds[:-1], bounds[1:]):
        xs = x[a:b].clone()   # its own allocation: a row slice of x is not 16-byte aligned in general
        v_last = torch.empty(N, dtype=torch.float32, device=H.DEV)
        s_seg, sv_seg, v_seg = H.layer.forward(cfg, xs, v_out=True, v_in=v_in, v_last=v_last)
        assert torch.equal(s_seg, spikes[a:b]), f"spikes of segment [{a}, {b})"
        assert torch.equal(v_seg, v[a:b]), f"membranes of segment [{a}, {b})"
        assert torch.equal(v_last, v[b - 1]), f"v_last of segment [{a}, {b})"
        states.append((a, b, xs, sv_seg, v_in))
        v_in = v_last
    g_in = None
    for a, b, xs, sv_seg, vi in reversed(states):
        g_out = torch.empty(N, dtype=torch.float32, device=H.DEV)
        gx_seg = H.layer.backward(cfg, xs, sv_seg, gs[a:b].clone(), v_in=vi, g_in=g_in, g_out=g_out)
        assert torch.equal(gx_seg, gx[a:b]), f"dL/dx of segment [{a}, {b})"
        assert torch.equal(g_out.to(gx.dtype), gx[a]), f"g_out of segment [{a}, {b})"
        g_in = g_out
    torch.cuda.synchronize()
    # the whole run itself against the oracle
    rep, _ = H.compare_layer(w, spikes, v, gx, x_np, gs_np)
    return rep


@pytest.mark.parametrize("T,N,lens", SPLITS, ids=lambda v: str(v))
@pytest.mark.parametrize("reset,io,spk", COMBOS, ids=lambda v: str(v))
def test_segments_equal_whole(H, T, N, lens, reset, io, spk):
    p = H.W.LifParams(0.5, 1.0, reset=reset)
    w = H.W.custom(f"seg{T}x{N}", T, N, p, seed=T + N, io=io, spk=spk, x_dist=("normal", 0.5, 0.5))
    rep = _segments_vs_whole(H, w, lens)
    assert rep.ok(), str(rep)
    H.torch.cuda.empty_cache()


@pytest.mark.parametrize("reset,io", list(itertools.product(["hard", "soft"], ["f32", "bf16"])))
def test_segment_from_arbitrary_state(H, reset, io):
    """v_in with values above and below V_th (spiking and not), NaN and +inf, and a
    nonzero g_in, against the oracle started from the same state."""
    torch = H.torch
    T, N = 37, 5003
    rng = np.random.default_rng(3)
    p = H.W.LifParams(0.75, 1.0, v_reset=0.125, alpha=2.0, reset=reset)
    w = H.W.custom("segstate", T, N, p, seed=9, io=io, x_dist=("normal", 0.3, 0.5))
    cfg = H.cfg_of(w)
    x_np, gs_np = H.W.x_full(w), H.W.gs_full(w)
    v_in = rng.normal(0.8, 0.6, size=N).astype(np.float32)
    v_in[:4] = [1.0, np.nextafter(np.float32(1.0), np.float32(0.0)), np.inf, np.nan]
    g_in = rng.normal(size=N).astype(np.float32)
    v_last = torch.empty(N, dtype=torch.float32, device=H.DEV)
    g_out = torch.empty(N, dtype=torch.float32, device=H.DEV)
    x, gs = H.to_dev(x_np, io), H.to_dev(gs_np, io)
    vi, gi = torch.from_numpy(v_in).to(H.DEV), torch.from_numpy(g_in).to(H.DEV)
    spikes, saved, v = H.layer.forward(cfg, x, v_out=True, v_in=vi, v_last=v_last)
    gx = H.layer.backward(cfg, x, saved, gs, v_in=vi, g_in=gi, g_out=g_out)
    torch.cuda.synchronize()

    op = H.oracle.Params.of(w.params)
    y_ref, v_ref = H.oracle.forward(op, x_np, v_init=v_in, y_init=(v_in >= np.float32(1.0)).astype(np.uint8))
    ref = H.oracle.backward(op, v_ref, y_ref, gs_np, g_next=g_in)
    y_gpu = H.parity.unpack_spikes(spikes.cpu().numpy(), N, w.spk)
    rep = H.parity.compare_forward(y_gpu, y_ref, v_ref, 1.0, v_gpu=v.cpu().numpy())
    H.parity.compare_grad(H.to_host_f32(gx), ref, io, rep)
    H.parity.compare_grad(g_out.cpu().numpy()[None, :], ref.sel(slice(0, 1)), "f32", rep)
    assert rep.ok(), str(rep)
    assert np.array_equal(v_last.cpu().numpy().view(np.uint32), v_ref[-1].view(np.uint32))


def test_segment_errors(H):
    torch = H.torch
    nat = H.native
    cfg = H.layer.LifConfig(0.5, 1.0)
    T, N = 4, 64
    x = torch.zeros((T, N), device=H.DEV)
    sp = torch.empty((T, N), dtype=torch.uint8, device=H.DEV)
    st = torch.zeros(N + 4, device=H.DEV)
    with pytest.raises(nat.SnnError) as e:
        nat.snn_lif_forward_seg(cfg.c(), T, N, x, st.data_ptr() + 4, sp, None)
    assert e.value.status == -4
    with pytest.raises(nat.SnnError) as e:
        nat.snn_lif_backward_seg(cfg.c(), T, N, x, None, None, x, st.data_ptr() + 4, x)
    assert e.value.status == -4
    # empty segments write nothing
    keep = torch.full((N,), 7.0, device=H.DEV)
    nat.snn_lif_forward_seg(cfg.c(), 0, N, None, None, None, None, keep)
    nat.snn_lif_backward_seg(cfg.c(), 0, N, None, None, None, None, None, None, keep)
    torch.cuda.synchronize()
    assert bool((keep == 7.0).all())


def _random_splits():
    """Seeded random cases: layer sizes on every plan (small, double-buffered, 1024-lane
    workgroups), 2-4 segments of random lengths, random hyper-parameters and formats."""
    rng = np.random.default_rng(20240803)
    sizes = [int(rng.integers(1, 5000)), int(rng.integers(60000, 80000)), int(rng.integers(500000, 700000)),
             2 * int(rng.integers(1 << 20, (1 << 21) + 500))]   # even: 2 neurons per lane, 1024-lane workgroups
    out = []
    for i in range(12):
        T = int(rng.integers(2, 91))
        N = sizes[i % len(sizes)]
        n_seg = int(rng.integers(2, min(4, T) + 1))
        cuts = np.sort(rng.choice(np.arange(1, T), size=n_seg - 1, replace=False))
        lens = [int(v) for v in np.diff(np.r_[0, cuts, T])]
        p = (float(rng.uniform(0, 1)), float(rng.uniform(0.2, 2.0)), float(rng.choice([0.0, rng.uniform(-0.5, 0.5)])),
             str(rng.choice(["hard", "soft"])))
        out.append((i, T, N, lens, p, str(rng.choice(["f32", "bf16"])), str(rng.choice(["u8", "bits", "io"]))))
    return out


@pytest.mark.parametrize("case", _random_splits(), ids=lambda c: f"rnd{c[0]}")
def test_random_segments_equal_whole(H, case):
    """Segments with the state handoff reproduce the single run bit for bit (the single run
    itself is checked against the oracle by the other parity tests)."""
    torch = H.torch
    i, T, N, lens, (decay, v_th, v_reset, reset), io, spk = case
    w = H.W.custom(f"rseg{i}", T, N, H.W.LifParams(decay, v_th, v_reset=v_reset, reset=reset), seed=700 + i, io=io,
                   spk=spk, x_dist=("normal", 0.5 * v_th, 0.5 * v_th + 0.2))
    cfg = H.cfg_of(w)
    x, gs = H.upload_rows(w, "x"), H.upload_rows(w, "gs")
    spikes, saved, v = H.layer.forward(cfg, x, v_out=True)
    gx = H.layer.backward(cfg, x, saved, gs)
    bounds = np.cumsum([0] + lens)
    states, v_in = [], None
    for a, b in zip(bounds[:-1], bounds[1:]):
        xs = x[a:b].clone()
        v_last = torch.empty(N, dtype=torch.float32, device=H.DEV)
        s_seg, sv_seg, v_seg = H.layer.forward(cfg, xs, v_out=True, v_in=v_in, v_last=v_last)
        assert torch.equal(s_seg, spikes[a:b]) and torch.equal(v_seg, v[a:b]), f"segment [{a}, {b}) of {lens}"
        states.append((a, b, xs, sv_seg, v_in))
        v_in = v_last
    g_in = None
    for a, b, xs, sv_seg, vi in reversed(states):
        g_out = torch.empty(N, dtype=torch.float32, device=H.DEV)
        gx_seg = H.layer.backward(cfg, xs, sv_seg, gs[a:b].clone(), v_in=vi, g_in=g_in, g_out=g_out)
        assert torch.equal(gx_seg.view(torch.uint8), gx[a:b].view(torch.uint8)), f"dL/dx of [{a}, {b}) of {lens}"
        g_in = g_out
    torch.cuda.synchronize()
    H.say(f"random segments {i}: T={T} N={N} {lens} {reset} {io} {spk}: equal")
    del x, gs, spikes, saved, v, gx, states
    torch.cuda.empty_cache()


def test_large_layer_as_segments_full_size(H):
    """The large bf16 layer at its full size (T = 256, N = 2^24, bit spikes): eight chained
    32-step segment calls give the single fused call's spikes and dL/dx bit for bit (the
    segments run single-chunk plans in 256-lane workgroups, the fused call the long-walk
    plan in 1024-lane workgroups)."""
    torch = H.torch
    T, N, S = 256, 1 << 24, 32
    cfg = H.layer.LifConfig(0.5, 1.0, io="bf16", spk="bits")
    c = cfg.c()
    gen = torch.Generator(device=H.DEV)
    gen.manual_seed(11)
    x = (torch.randn((T, N), device=H.DEV, generator=gen) * 0.5 + 0.5).to(torch.bfloat16)
    gs = torch.randn((T, N), device=H.DEV, generator=gen).to(torch.bfloat16)
    spikes, saved, _ = H.layer.forward(cfg, x)
    gx = H.layer.backward(cfg, x, saved, gs)
    torch.cuda.synchronize()
    del saved
    seg_spikes = torch.empty_like(spikes)
    seg_gx = torch.empty_like(gx)
    v_last = torch.empty((T // S, N), dtype=torch.float32, device=H.DEV)
    g = [torch.empty(N, dtype=torch.float32, device=H.DEV) for _ in range(2)]
    assert H.native.snn_lif_saved_bytes(c, S, N) == 0
    for s in range(T // S):
        H.native.snn_lif_forward_seg(c, S, N, x[s * S], v_last[s - 1] if s else None, seg_spikes[s * S], None,
                                     v_last[s], None)
    for i, s in enumerate(range(T // S - 1, -1, -1)):
        H.native.snn_lif_backward_seg(c, S, N, x[s * S], v_last[s - 1] if s else None, None, gs[s * S],
                                      g[i % 2] if i else None, seg_gx[s * S], g[(i + 1) % 2])
    torch.cuda.synchronize()
    assert torch.equal(seg_spikes, spikes)
    assert torch.equal(seg_gx.view(torch.int16), gx.view(torch.int16))
    del x, gs, gx, seg_gx, spikes, seg_spikes
    torch.cuda.empty_cache()
