"""Seeded random configurations against the oracle: sizes (log-uniform N up to 2^18, T up
to 80), reset, I/O dtype, spike format and hyper-parameters (decay in [0, 1], threshold
and reset value of either sign, surrogate sharpness) drawn from a fixed generator, so the
combinations the structured tests do not list are covered too.  Every case runs in full
on both sides.  A second set draws large layers (2M-4.2M neurons, 17-80 steps: several
chunks in 1024-lane workgroups), run in full on the GPU and checked on sampled columns."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

N_CASES = 60


def _cases():
    rng = np.random.default_rng(20240801)
    out = []
    for i in range(N_CASES):
        T = int(rng.integers(1, 81))
        N = int(np.exp(rng.uniform(0, np.log(1 << 18))))
        decay = float(rng.choice([0.0, 0.2, 0.5, 0.9, 1.0, rng.uniform(0, 1)]))
        v_th = float(rng.uniform(-0.5, 2.0))
        v_reset = float(rng.choice([0.0, rng.uniform(-0.5, 1.0)]))
        alpha = float(rng.uniform(0.5, 8.0))
        reset = str(rng.choice(["hard", "soft"]))
        io = str(rng.choice(["f32", "bf16"]))
        spk = str(rng.choice(["u8", "bits", "io"]))
        out.append((i, T, N, decay, v_th, v_reset, alpha, reset, io, spk))
    return out


@pytest.fixture(scope="module")
def H():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_harness
    return gpu_harness


@pytest.mark.parametrize("case", _cases(), ids=lambda c: f"case{c[0]}")
def test_random_config(H, case):
    i, T, N, decay, v_th, v_reset, alpha, reset, io, spk = case
    p = H.W.LifParams(decay, v_th, v_reset=v_reset, alpha=alpha, reset=reset)
    scale = abs(v_th) + 0.5
    w = H.W.custom(f"rnd{i}", T, N, p, seed=500 + i, io=io, spk=spk, x_dist=("normal", 0.4 * v_th, 0.6 * scale))
    rep = H.check_full(w)
    assert rep.ok(), f"T={T} N={N} decay={decay} v_th={v_th} v_reset={v_reset} alpha={alpha} {reset} {io} {spk}: {rep}"


N_LARGE = 12


def _large_cases():
    rng = np.random.default_rng(20240802)
    out = []
    for i in range(N_LARGE):
        T = int(rng.integers(17, 81))
        N = int(rng.integers(1 << 21, (1 << 22) + (1 << 17)))
        N -= N % 2 if rng.random() < 0.8 else 0       # mostly even N (2 neurons per lane)
        decay = float(rng.uniform(0, 1))
        v_th = float(rng.uniform(-0.5, 2.0))
        v_reset = float(rng.choice([0.0, rng.uniform(-0.5, 1.0)]))
        alpha = float(rng.uniform(0.5, 8.0))
        reset = str(rng.choice(["hard", "soft"]))
        io = str(rng.choice(["f32", "bf16"]))
        spk = str(rng.choice(["u8", "bits", "io"]))
        out.append((i, T, N, decay, v_th, v_reset, alpha, reset, io, spk))
    return out


@pytest.mark.parametrize("case", _large_cases(), ids=lambda c: f"large{c[0]}")
def test_random_large_config(H, case):
    i, T, N, decay, v_th, v_reset, alpha, reset, io, spk = case
    p = H.W.LifParams(decay, v_th, v_reset=v_reset, alpha=alpha, reset=reset)
    scale = abs(v_th) + 0.5
    w = H.W.custom(f"rndL{i}", T, N, p, seed=900 + i, io=io, spk=spk, x_dist=("normal", 0.4 * v_th, 0.6 * scale))
    rep = H.check_sampled(w, 1 << 12, v_out=True)
    H.say(f"random large {i}: T={T} N={N} {reset} {io} {spk}: {rep}")
    assert rep.ok(), f"T={T} N={N} decay={decay} v_th={v_th} v_reset={v_reset} alpha={alpha} {reset} {io} {spk}: {rep}"
    H.torch.cuda.empty_cache()
