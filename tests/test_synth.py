"""The seeded input generator: index-addressable, deterministic, right distributions.  CPU only."""
import numpy as np

import synth
from synth import workloads as W


def test_subset_matches_full_tensor():
    w = W.custom("t", 7, 1000, W.HARD_05, x_dist=("normal", 0.5, 0.5), burst=(0.1, 1.5))
    full = W.x_full(w)
    cols = np.array([0, 3, 999, 512, 17])
    assert np.array_equal(W.x_cols(w, cols), full[:, cols])
    assert np.array_equal(W.x_rows(w, 2, 5), full[2:5])
    assert np.array_equal(W.gs_cols(w, cols), W.gs_full(w)[:, cols])


def test_bf16_rounding_and_widening():
    a = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -0.0, np.inf, 3.14159265], dtype=np.float32)
    b = synth.bf16_bits_to_f32(synth.to_bf16_bits(a))
    # ties go to even: 1 + 2^-8 -> 1, 1 + 3*2^-8 -> 1 + 2^-6
    assert b.tolist()[:3] == [1.0, 1.0, 1.0 + 2 ** -6]
    assert np.signbit(b[3]) and b[4] == np.inf
    assert abs(b[5] - 3.140625) == 0
    nan = synth.to_bf16_bits(np.array([np.nan], dtype=np.float32))
    assert np.isnan(synth.bf16_bits_to_f32(nan))[0]


def test_distributions():
    n = 1 << 20
    z = synth.fill(3, 0, ("normal", 0.0, 1.0), n)
    assert abs(z.mean()) < 5e-3 and abs(z.std() - 1) < 5e-3
    assert abs(np.mean(z ** 4) - 3) < 0.05           # Gaussian kurtosis
    u = synth.fill(3, 1, ("uniform", 0.5, 2.0), n)
    assert u.min() >= 0.5 and u.max() <= 2.0 and abs(u.mean() - 1.25) < 5e-3
    m = np.zeros(n, dtype=np.float32)
    synth.bernoulli_set(3, 2, 0.1, 1.0, m)
    assert abs(m.mean() - 0.1) < 2e-3


def test_streams_and_seeds_differ():
    a = synth.fill(1, 0, ("normal", 0, 1), 64)
    assert not np.array_equal(a, synth.fill(1, 1, ("normal", 0, 1), 64))
    assert not np.array_equal(a, synth.fill(2, 0, ("normal", 0, 1), 64))
    assert np.array_equal(a, synth.fill(1, 0, ("normal", 0, 1), 64))
    assert synth.bits(1, 0, 5) != synth.bits(1, 0, 6)


def test_workload_shapes():
    assert W.WORKLOADS["conv"].N == 64 * 128 * 32 * 32
    assert W.WORKLOADS["long"].N == 32 * 4096 and W.WORKLOADS["long"].params.reset == "soft"
    assert W.WORKLOADS["stack"].layers == 3 and W.WORKLOADS["stack"].F == 4096
    assert W.WORKLOADS["large"].N == 1 << 24 and W.WORKLOADS["large"].io == "bf16"
