"""The synthetic-input generator: distribution, determinism and window indexing."""

import numpy as np

import synth
from synth import gen


def test_normal_moments_and_support():
    x = synth.normal_f32(0, 2, np.arange(400_000), std=0.0316)
    assert x.dtype == np.float32
    assert abs(x.mean()) < 4 * 0.0316 / np.sqrt(x.size)
    assert abs(x.std() / 0.0316 - 1.0) < 0.01
    assert np.abs(x).max() <= 3.47 * 0.0316
    # excess kurtosis of a 4-term Irwin-Hall sum is -0.3 (close to normal)
    k = ((x - x.mean()) ** 4).mean() / x.var() ** 2 - 3.0
    assert abs(k + 0.3) < 0.05


def test_uniform_range():
    u = synth.uniform_f32(1, 3, np.arange(100_000), half_width=0.5)
    assert u.min() >= -0.5 and u.max() < 0.5
    assert abs(u.mean()) < 0.01


def test_streams_and_windows_are_consistent():
    full = synth.normal_f32(7, 1, np.arange(3 * 50), std=1.0).reshape(3, 50)
    win = synth.normal_f32(7, 1, gen.window_index(3, 50, 10, 17), std=1.0).reshape(3, 7)
    np.testing.assert_array_equal(full[:, 10:17], win)
    other = synth.normal_f32(7, 2, np.arange(150), std=1.0)
    assert not np.array_equal(full.reshape(-1), other)


def test_splitmix_reference_values():
    # SplitMix64 seeded with state 0 produces 0xE220A8397B1DCDAF first (the
    # generator's published reference output, e.g. in Vigna's splitmix64.c)
    assert gen._fmix_int(0 + gen.GAMMA) == 0xE220A8397B1DCDAF
    w = synth.splitmix_words(0, 0, [0, 1])
    key = synth.splitmix_key(0, 0)
    assert int(w[0]) == gen._fmix_int(key + gen.GAMMA)
    assert int(w[1]) == gen._fmix_int(key + 2 * gen.GAMMA)
