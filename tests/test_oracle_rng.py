"""Pins of the oracle's counter-based generator and synthetic-data recipe.

The generator is SplitMix64 (Steele, Lea & Flood, OOPSLA 2014); the random
minibatch of Algorithm 1 (Sec. 3.1) is read as i.i.d. draws with replacement
(Sec. 2 makes the samples i.i.d. realisations).
"""

import os

import numpy as np
import pytest

from oracle import rng

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_hex(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [int(line, 16) for line in f if line.strip() and not line.startswith("#")]


def test_splitmix64_published_sequence():
    want = _golden_hex("splitmix64_seed0.txt")
    assert rng.splitmix64_sequence(0, len(want)) == want


def test_counter_form_equals_sequence():
    # H(key, c) is the (c+1)-th output of the generator started at `key`.
    for key in (0, 1, 0xDEADBEEFCAFEF00D):
        seq = rng.splitmix64_sequence(key, 9)
        assert [rng.h_scalar(key, c) for c in range(9)] == seq


def test_vectorised_hash_matches_scalar():
    r = np.random.default_rng(7)
    keys = [int(k) for k in r.integers(0, 2**63, size=3, dtype=np.int64)] + [2**64 - 1]
    ctr = r.integers(0, 2**63, size=200, dtype=np.int64).astype(np.uint64)
    ctr[:3] = [0, 2**64 - 1, 2**32]
    for key in keys:
        got = rng.h(key, ctr)
        want = np.array([rng.h_scalar(key, int(c)) for c in ctr], dtype=np.uint64)
        assert np.array_equal(got, want)


def test_index_draw_bit_fields_brute_force():
    seed, N = 11, 50000
    key = rng.stream_key(seed, rng.TAG_INDEX)
    for (j, t, B) in [(0, 0, 5), (3, 7, 9), (65535, 2**31, 3)]:
        got = rng.draw_indices(seed, j, t, B, N)
        want = [rng.h_scalar(key, (t << 32) | (j << 16) | s) % N for s in range(B)]
        assert got.tolist() == want
    # the draw of sample s does not depend on the batch size (fixed bit fields)
    assert np.array_equal(rng.draw_indices(seed, 2, 5, 4, N), rng.draw_indices(seed, 2, 5, 64, N)[:4])


def test_index_draw_uniform_chi2():
    N, B = 64, 4096
    draws = np.concatenate([rng.draw_indices(3, j, t, B, N) for j in range(4) for t in range(4)])
    counts = np.bincount(draws, minlength=N)
    expect = len(draws) / N
    chi2 = float(((counts - expect) ** 2 / expect).sum())
    # 63 degrees of freedom: mean 63, sd ~11.2; 120 is ~5 sd
    assert chi2 < 120.0
    assert draws.min() >= 0 and draws.max() < N


def test_normal_surrogate_exact_and_moments():
    key = rng.stream_key(5, rng.TAG_NOISE)
    e = np.arange(200000, dtype=np.uint64)
    z = rng.normal_surrogate(key, e)
    # exactly representable in float32, bounded by the Irwin-Hall support
    assert np.array_equal(z.astype(np.float32).astype(np.float64), z)
    assert np.abs(z).max() <= 393210 / 65536
    assert abs(z.mean()) < 5 * (1 / np.sqrt(len(z)))
    assert abs(z.var() - 1.0) < 5 * np.sqrt(2.0 / len(z))
    # brute force of the definition for a few counters
    for ei in (0, 1, 12345):
        fields = 0
        for r in range(3):
            v = rng.h_scalar(key, 3 * ei + r)
            fields += sum((v >> (16 * f)) & 0xFFFF for f in range(4))
        assert z[ei] == (fields - 393210) / 65536.0


def test_dataset_rows_recipe():
    seed, IN, C, sigma = 4, 16, 3, 0.5
    rows = np.arange(3000)
    X, y = rng.data_rows(seed, rows, IN, C, sigma)
    assert np.array_equal(X.astype(np.float32).astype(np.float64), X)
    assert set(np.unique(y).tolist()) == {0, 1, 2}
    mu = rng.class_means(seed, np.arange(C), IN)
    for c in range(C):
        resid = X[y == c] - mu[c]
        assert abs(resid.std() - sigma) < 0.03
        assert np.abs(resid.mean(axis=0)).max() < 0.1
    # one element written out from the definition
    i, d = 17, 5
    z = rng.normal_surrogate(rng.stream_key(seed, rng.TAG_NOISE), np.array([i * IN + d], dtype=np.uint64))[0]
    assert X[i, d] == float(np.float32(mu[y[i], d] + sigma * z))
    assert y[i] == rng.h_scalar(rng.stream_key(seed, rng.TAG_LABEL), i) % C


def test_initial_weights_recipe():
    W = rng.init_uniform(9, 1, 7, 33)
    s = float(np.float32(1 / np.sqrt(33.0)))
    assert np.abs(W).max() <= s
    key = rng.stream_key(9, rng.TAG_INIT)
    o, i = 4, 30
    u = (rng.h_scalar(key, (1 << 48) + o * 33 + i) >> 40) * 2.0 ** -24
    assert W[o, i] == float(np.float32((2 * u - 1) * s))


@pytest.mark.parametrize("std", [0.01, 0.3])
def test_given_gradients_scale(std):
    g = rng.given_gradients(2, 3, 5, 100000, std)
    assert abs(g.std() / np.float32(std) - 1.0) < 0.02
    assert np.array_equal(g.astype(np.float32).astype(np.float64), g)
