"""Pins of the p-less oracle (the truncation rule of the cited p-less paper:
keep p_i >= sum_j p_j^2 of softmax(z / T), then one inverse-CDF draw in
ascending id order): closed forms worked out by hand, the two-token and
uniform special cases, invariants, an agreement-probability simulation of the
threshold, and the draw distribution."""
import math

import numpy as np
import pytest

from oracle import philox
from oracle import pless


def _logits(p, T=1.0):
    return np.log(np.asarray(p, np.float64)) * T


def test_worked_examples():
    # p = (1/2, 1/4, 1/8, 1/8): sum p^2 = 1/4 + 1/16 + 2/64 = 0.34375 -> only token 0
    p, thr, kept = pless.pless_probabilities(_logits([0.5, 0.25, 0.125, 0.125]), 1.0)
    assert thr == pytest.approx(0.34375, rel=1e-12)
    assert list(np.flatnonzero(kept)) == [0]
    # p = (0.4, 0.2, 0.2, 0.1, 0.1): sum p^2 = 0.26 -> only token 0
    _, thr, kept = pless.pless_probabilities(_logits([0.4, 0.2, 0.2, 0.1, 0.1]), 1.0)
    assert thr == pytest.approx(0.26, rel=1e-12)
    assert list(np.flatnonzero(kept)) == [0]
    # p = (0.1, 0.3, 0.2, 0.3, 0.1): sum p^2 = 0.24 -> tokens 1 and 3, W = 0.6,
    # C = (0.3, 0.6): u < 1/2 draws 1, u >= 1/2 draws 3
    z = _logits([0.1, 0.3, 0.2, 0.3, 0.1])
    _, thr, kept = pless.pless_probabilities(z, 1.0)
    assert thr == pytest.approx(0.24, rel=1e-12)
    assert list(np.flatnonzero(kept)) == [1, 3]
    assert [pless.sample_pless(z, 1.0, u).token for u in (0.0, 0.3, 0.49, 0.51, 0.99)] == [1, 1, 1, 3, 3]


def test_temperature_scales_logits_first():
    # z = 2 ln p at T = 2 is p = (0.35, 0.25, 0.2, 0.1, 0.1): sum p^2 = 0.245 keeps
    # tokens 0 and 1.  Truncating softmax(z) first (prop. to p^2, sum of squares
    # 0.345) would keep token 0 alone.
    z = _logits([0.35, 0.25, 0.2, 0.1, 0.1], T=2.0)
    _, thr, kept = pless.pless_probabilities(z, 2.0)
    assert thr == pytest.approx(0.245, rel=1e-12)
    assert list(np.flatnonzero(kept)) == [0, 1]
    _, _, kept1 = pless.pless_probabilities(z, 1.0)
    assert list(np.flatnonzero(kept1)) == [0]


def test_uniform_keeps_everything():
    # p = 1/8 everywhere: sum p^2 = 1/8 exactly, every token on the edge and kept
    for T in (0.5, 1.0, 3.0):
        z = np.full(8, 1.7)
        p, thr, kept = pless.pless_probabilities(z, T)
        assert thr == 0.125 and kept.all()
        for u in (0.01, 0.3, 0.6, 0.99):
            assert pless.sample_pless(z, T, u).token == math.floor(8 * u)


def test_two_tokens_keep_only_the_more_probable():
    # p2 >= p1^2 + p2^2 <=> p2 * p1 >= p1^2 <=> p2 >= p1: one survivor unless tied
    g = np.random.default_rng(5)
    for _ in range(200):
        z = g.normal(size=2) * 3
        if abs(z[0] - z[1]) < 1e-9:
            continue
        _, _, kept = pless.pless_probabilities(z, float(g.uniform(0.3, 3)))
        assert list(np.flatnonzero(kept)) == [int(np.argmax(z))]


def test_k_tied_top_tokens_and_a_light_tail():
    # k tokens at p = a and the rest tiny: sum p^2 ~ k a^2 < a, the k survive
    V, k = 1000, 5
    z = np.full(V, -20.0)
    top = [3, 100, 555, 700, 999]
    z[top] = 0.0
    _, thr, kept = pless.pless_probabilities(z, 1.0)
    assert sorted(np.flatnonzero(kept)) == top
    assert thr == pytest.approx(1 / k, rel=1e-5)


def test_argmax_always_kept_and_shift_invariance():
    g = np.random.default_rng(7)
    for _ in range(50):
        z = g.normal(size=int(g.integers(2, 3000))) * g.uniform(0.1, 5)
        T = float(g.uniform(0.2, 4))
        p, thr, kept = pless.pless_probabilities(z, T)
        assert kept[np.argmax(z)]
        assert thr <= p.max() + 1e-15
        p2, thr2, kept2 = pless.pless_probabilities(z + 123.25, T)
        assert np.array_equal(kept, kept2) and thr2 == pytest.approx(thr, rel=1e-12)


def test_small_temperature_is_argmax():
    g = np.random.default_rng(11)
    for _ in range(20):
        z = g.normal(size=500)
        for u in (0.0, 0.5, 0.999):
            assert pless.sample_pless(z, 1e-3, u).token == int(np.argmax(z))
    assert pless.sample_pless(np.array([1.0, 5.0, 5.0]), 0.0, 0.7).token == 1


def test_threshold_is_the_agreement_probability_of_two_draws():
    # sum p^2 is the chance that two independent draws agree: simulate it
    g = np.random.default_rng(13)
    z = g.normal(size=40) * 1.5
    p, thr, _ = pless.pless_probabilities(z, 1.3)
    n = 400_000
    a = g.choice(40, size=n, p=p)
    b = g.choice(40, size=n, p=p)
    agree = float(np.mean(a == b))
    assert abs(agree - thr) < 5 * math.sqrt(thr * (1 - thr) / n)


def test_inverse_cdf_matches_searchsorted_and_many_matches_single():
    g = np.random.default_rng(17)
    z = g.normal(size=5000) * 2
    T = 1.7
    w = pless.kept_probabilities(z, T)
    cdf = np.cumsum(w)
    us = philox.uniform(99, 0, np.arange(300, dtype=np.uint64))
    many = pless.sample_pless_many(z, T, us)
    for u, d in zip(us, many):
        one = pless.sample_pless(z, T, float(u))
        assert one.token == d.token
        if d.cdf_margin > 1e-9:
            assert d.token == int(np.searchsorted(cdf, float(u), side="right"))


def test_draw_on_an_exact_running_sum():
    """The draw takes the first kept token whose running sum is strictly above
    u * W: with equal probabilities the running sums are exact multiples of
    1/n, and u on such an edge selects the next token (both draw forms)."""
    z2 = np.zeros(2)
    for u, want in ((0.5, 1), (0.0, 0), (0.75, 1), (0.25, 0)):
        assert pless.sample_pless(z2, 1.0, u).token == want
        assert pless.sample_pless_many(z2, 1.0, [u])[0].token == want
    us = [0.25, 0.5, 0.75, 0.0]
    assert [pless.sample_pless(np.zeros(4), 1.0, u).token for u in us] == [1, 2, 3, 0]
    assert [d.token for d in pless.sample_pless_many(np.zeros(4), 1.0, us)] == [1, 2, 3, 0]


def test_draw_distribution_chi_square():
    from scipy import stats
    g = np.random.default_rng(19)
    z = np.concatenate([g.normal(size=12) + 3.0, g.normal(size=3000)])
    T = 2.0
    q = pless.kept_probabilities(z, T)
    support = np.flatnonzero(q > 0)
    D = 20000
    us = philox.uniform(7, 0, np.arange(D, dtype=np.uint64))
    toks = np.array([d.token for d in pless.sample_pless_many(z, T, us)])
    assert set(np.unique(toks)) <= set(support)
    obs = np.bincount(toks, minlength=len(z))[support]
    assert stats.chisquare(obs, q[support] * D).pvalue > 1e-4


def test_margins_reported():
    z = _logits([0.1, 0.3, 0.2, 0.3, 0.1])
    d = pless.sample_pless(z, 1.0, 0.5)           # u * W lands on the edge C_1 = 0.3
    assert d.cdf_margin < 1e-12
    # the nearest mask decision is token 2 (p = 0.2 against 0.24)
    assert d.logit_margin == pytest.approx(math.log(0.24) - math.log(0.2), rel=1e-9)
