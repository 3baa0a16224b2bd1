"""Pins for the oracle's argmax and min-p sampler (not GPU)."""
import math

import numpy as np
import pytest
from scipy import special, stats

from oracle import sampler


def test_argmax_first_index_on_ties():
    z = np.array([0.5, 3.0, -1.0, 3.0, 2.0])
    assert sampler.argmax(z) == 1
    assert sampler.sample_minp(z, 0.0, 0.1, 0.7).token == 1


@pytest.mark.parametrize("u", [0.0, 0.3, 0.999999])
def test_small_temperature_reduces_to_argmax(u):
    g = np.random.default_rng(1)
    z = g.normal(size=1000)
    z[417] = z.max() + 0.5          # unique max with a clear gap
    assert sampler.sample_minp(z, 1e-3, 0.05, u).token == 417


@pytest.mark.parametrize("T,p_min", [(0.7, 0.05), (1.0, 0.1), (2.0, 0.2), (3.0, 0.05)])
def test_minp_kept_set_matches_explicit_softmax(T, p_min):
    g = np.random.default_rng(int(T * 10 + p_min * 100))
    z = g.normal(size=5000) * 2
    p = special.softmax(z / T)
    want = p >= p_min * p.max()
    _, kept = sampler.minp_weights(z, T, p_min)
    assert np.array_equal(kept, want)


@pytest.mark.parametrize("seed", range(5))
def test_inverse_cdf_matches_searchsorted(seed):
    g = np.random.default_rng(seed)
    z = g.normal(size=3000)
    T, p_min = 1.5, 0.1
    p = special.softmax(z / T)
    kept = p >= p_min * p.max()
    pk = np.where(kept, p, 0.0)
    for u in g.random(50):
        want = int(np.searchsorted(np.cumsum(pk), u * pk.sum(), side="right"))
        assert sampler.sample_minp(z, T, p_min, u).token == want


def test_brute_force_interval_measure_tiny():
    """On a 5-token row, the set of u mapping to token i has measure equal to
    its kept probability (u scanned on a fine grid)."""
    z = np.array([1.0, 2.0, -3.0, 1.5, 0.2])
    T, p_min = 1.0, 0.2
    grid = (np.arange(1 << 16) + 0.5) / (1 << 16)
    toks = np.array([sampler.sample_minp(z, T, p_min, u).token for u in grid])
    freq = np.bincount(toks, minlength=5) / grid.size
    e = np.exp(z - z.max())
    p_manual = np.where(e >= p_min, e, 0) / np.where(e >= p_min, e, 0).sum()
    assert np.allclose(freq, p_manual, atol=2.0 / grid.size)
    assert freq[2] == 0 and freq[4] == 0     # exp(-5), exp(-1.8) < 0.2


def test_pmin_one_is_argmax_and_pmin_zero_is_full_softmax():
    g = np.random.default_rng(3)
    z = g.normal(size=200)
    for u in (0.01, 0.5, 0.99):
        assert sampler.sample_minp(z, 2.0, 1.0, u).token == int(np.argmax(z))
    probs = sampler.kept_probabilities(z, 2.0, 1e-300)
    assert np.allclose(probs, special.softmax(z / 2.0), rtol=1e-12, atol=0)


def test_draw_distribution_chi_square():
    g = np.random.default_rng(9)
    z = g.normal(size=40) * 1.5
    T, p_min = 1.0, 0.1
    probs = sampler.kept_probabilities(z, T, p_min)
    u = g.random(40000)
    toks = np.array([sampler.sample_minp(z, T, p_min, x).token for x in u])
    support = np.flatnonzero(probs > 0)
    assert set(np.unique(toks)) <= set(support)
    obs = np.bincount(toks, minlength=z.size)[support]
    assert stats.chisquare(obs, probs[support] * u.size).pvalue > 1e-4


def test_margins_reported():
    z = np.array([0.0, math.log(0.1) * 2.0])      # second logit exactly at the min-p edge (T=2)
    d = sampler.sample_minp(z, 2.0, 0.1, 0.25)
    assert d.logit_margin < 1e-12
    d = sampler.sample_minp(np.array([0.0, 0.0]), 1.0, 0.1, 0.5)   # u*W on the CDF edge
    assert d.cdf_margin == 0.0 and d.token == 1


def test_many_matches_single():
    g = np.random.default_rng(21)
    z = g.normal(size=700) * 2
    us = g.random(300)
    many = sampler.sample_minp_many(z, 1.3, 0.07, us)
    for u, d in zip(us, many):
        one = sampler.sample_minp(z, 1.3, 0.07, u)
        assert d.token == one.token
        assert np.isclose(d.cdf_margin, one.cdf_margin, rtol=0, atol=1e-15)


def test_draw_on_an_exact_running_sum():
    """The draw returns the smallest kept id whose running kept-weight sum
    exceeds u * W (strictly): with two equal weights (W = 2) and u = 0.5 the
    target 1.0 equals the first running sum, so token 1 is drawn, and u = 0
    draws token 0.  The one-draw and many-draw forms agree on these edges."""
    z = np.zeros(2)
    for u, want in ((0.5, 1), (0.0, 0), (0.75, 1), (0.25, 0)):
        assert sampler.sample_minp(z, 1.0, 0.1, u).token == want
        assert sampler.sample_minp_many(z, 1.0, 0.1, [u])[0].token == want
    z3 = np.zeros(4)                                   # W = 4, edges at 1, 2, 3
    us = [0.25, 0.5, 0.75, 0.0]
    assert [d.token for d in sampler.sample_minp_many(z3, 1.0, 0.1, us)] == [1, 2, 3, 0]
    assert [sampler.sample_minp(z3, 1.0, 0.1, u).token for u in us] == [1, 2, 3, 0]
