"""Pins of the oracle's generator and pattern sampler (Sec. III-D, Eqs. 2-3)."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

from oracle import prng, search

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix64_published_sequence():
    g = json.load(open(os.path.join(GOLDEN, "splitmix64_state0.json")))
    state = int(g["initial_state"], 16)
    for want in g["outputs"]:
        state, out = prng.splitmix64_next(state)
        assert out == int(want, 16)


def test_counter_stream_state_layout():
    # seed 0, stream 0, iteration 0 is the plain sequence from state 0
    g = json.load(open(os.path.join(GOLDEN, "splitmix64_state0.json")))
    s = prng.CounterStream(0, 0, 0)
    assert s.next_u64() == int(g["outputs"][0], 16)
    # stream and iteration enter by XOR into disjoint bit fields
    assert prng.CounterStream(5, 3, 7).state == 5 ^ ((3 << 40) | 7)
    with pytest.raises(ValueError):
        prng.CounterStream(0, 1 << 24, 0)
    with pytest.raises(ValueError):
        prng.CounterStream(0, 0, 1 << 40)


def test_uniform_distribution_ks():
    s = prng.CounterStream(1805, 1, 0)
    u = np.array([s.next_uniform() for _ in range(100_000)])
    assert u.min() >= 0.0 and u.max() < 1.0
    assert stats.kstest(u, "uniform").pvalue > 1e-3


@pytest.mark.parametrize("n", [1, 3, 7, 16])
def test_next_below_unbiased(n):
    s = prng.CounterStream(8939, 2, 5)
    x = np.array([s.next_below(n) for _ in range(60_000)])
    assert x.min() >= 0 and x.max() < n
    if n > 1:
        counts = np.bincount(x, minlength=n)
        assert stats.chisquare(counts).pvalue > 1e-3


def test_sample_period_inverse_cdf_edges():
    K = [0.25, 0.25, 0.5]
    assert prng.sample_period(K, 0.0) == 1
    assert prng.sample_period(K, 0.2499999) == 1
    assert prng.sample_period(K, 0.25) == 2        # strict u < C_i
    assert prng.sample_period(K, 0.5) == 3
    assert prng.sample_period(K, 0.9999999) == 3
    # rounding leaves no C_i above u: fall back to the last positive entry
    assert prng.sample_period([0.5, 0.25, 0.0], 0.9) == 2
    for i in range(5):
        e = [0.0] * 5
        e[i] = 1.0
        assert prng.sample_period(e, 0.7) == i + 1


def test_sampler_period_frequencies_follow_K():
    K = search.closed_form(0.5, 16)
    draws = [prng.sample_row_pattern(K, 8939, 0, it) for it in range(40_000)]
    periods = np.array([d[0] for d in draws])
    counts = np.bincount(periods, minlength=17)[1:]
    expected = K * len(draws)
    keep = expected > 5
    chi = stats.chisquare(counts[keep], expected[keep] * counts[keep].sum() / expected[keep].sum())
    assert chi.pvalue > 1e-3
    for p, o in draws[:2000]:
        assert 0 <= o < p


def test_eq2_per_neuron_drop_probability_exact():
    """Eq. 2: every neuron is dropped with probability sum_i k_i (i-1)/i.

    Enumerate the sampler's outcomes (period i with probability k_i, offset
    uniform on {0..i-1}) in exact rational arithmetic.
    """
    K = [Fraction(1, 10), Fraction(2, 10), Fraction(3, 10), Fraction(4, 10)]
    target = sum(k * Fraction(i - 1, i) for i, k in enumerate(K, start=1))
    for j in range(60):
        pd = Fraction(0)
        for i, k in enumerate(K, start=1):
            for o in range(i):
                if j % i != o:
                    pd += k * Fraction(1, i)
        assert pd == target


@pytest.mark.parametrize("p", [0.3, 0.5, 0.7])
def test_empirical_per_neuron_drop_rate(p):
    """Over 1e5 sampled patterns each neuron's drop frequency is within 0.01 of p."""
    K = search.distribution_for_rate(p, 16)
    n_neurons = 2048
    pair_counts = {}
    n_draws = 100_000
    for it in range(n_draws):
        key = prng.sample_row_pattern(K, 8939, 1, it)
        pair_counts[key] = pair_counts.get(key, 0) + 1
    kept = np.zeros(n_neurons)
    j = np.arange(n_neurons)
    for (per, off), c in pair_counts.items():
        kept += c * (j % per == off)
    rate = 1.0 - kept / n_draws
    assert np.max(np.abs(rate - p)) < 0.01


def test_tdp_bitmap_rule():
    words = prng.tile_bitmap_tdp(3, 5, 4, 1)
    bits = [(words[t // 32] >> (t % 32)) & 1 for t in range(15)]
    assert bits == [1 if t % 4 == 1 else 0 for t in range(15)]


def test_bernoulli_bitmap_extremes_and_rate():
    ones = prng.tile_bitmap_bernoulli(8, 8, 0.0, 1, 0, 0)
    assert all(w == 0xFFFFFFFF for w in ones)
    zeros = prng.tile_bitmap_bernoulli(8, 8, 1.0, 1, 0, 0)
    assert all(w == 0 for w in zeros)
    words = prng.tile_bitmap_bernoulli(64, 64, 0.5, 8939, 0, 0)
    kept = sum(bin(w).count("1") for w in words)
    # binomial(4096, 0.5): 6 sigma = 192
    assert abs(kept - 2048) < 192
