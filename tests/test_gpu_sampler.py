"""Sampler and argmax kernels vs the oracle on identical fp32 logits (the
sampler sweep workload: V=152064, 256 rows, Zipf-biased logits)."""
import numpy as np
import pytest

import synth
from oracle import philox, sampler
from tests.gpu_common import Tally, argmax_gpu, judge_draw, sample_gpu

pytestmark = pytest.mark.gpu
MARGIN = 1e-4


@pytest.fixture(scope="module")
def rgd():
    import paper_2607_20791_amd as m
    return m


@pytest.fixture(scope="module")
def z():
    return synth.sweep_logits()


def test_argmax_matches_oracle(rgd, z):
    got = argmax_gpu(rgd, z)
    want = np.array([sampler.argmax(r) for r in z])
    assert np.array_equal(got, want)


def test_argmax_ties_lowest_index(rgd):
    g = np.random.default_rng(3)
    z = g.normal(size=(5, 9000)).astype(np.float32)
    for r, pos in enumerate([(0, 7), (100, 8191), (4095, 4096), (8999, 3), (10, 20, 8998)]):
        for p in pos:
            z[r, p] = 50.0
    got = argmax_gpu(rgd, z)
    assert list(got) == [0, 100, 4095, 3, 10]


@pytest.mark.parametrize("V", [1, 5, 1003, 4097, 8193])
def test_argmax_any_vocab(rgd, V):
    """Vocabularies that are not a multiple of 4 (unaligned rows) take the
    scalar path; the last position and ties across chunk edges included."""
    g = np.random.default_rng(V)
    z = g.normal(size=(3, V)).astype(np.float32)
    z[1, V - 1] = 40.0
    if V > 4096:
        z[2, 4095] = z[2, 4096] = 41.0
    got = argmax_gpu(rgd, z)
    want = np.array([sampler.argmax(r) for r in z])
    assert np.array_equal(got, want)


def _check_rows(name, z, T, pmin, got, seeds, ctr, stream):
    tally = Tally(name)
    for r in range(got.shape[0]):
        u = float(philox.uniform(int(seeds[r]), ctr, stream))
        tally.add(judge_draw(z[r], T, pmin, u, int(got[r])))
    return tally.close()


@pytest.mark.parametrize("T", synth.SWEEP.temperatures)
@pytest.mark.parametrize("pmin", synth.SWEEP.min_ps)
def test_minp_single_draw_grid(rgd, z, T, pmin):
    rows = z[:48]
    seeds = np.arange(48, dtype=np.uint64)
    got = sample_gpu(rgd, rows, T, pmin, seeds, ctr=0, stream0=0, draws=1)[:, 0]
    _check_rows(f"sampler sweep, 48 rows, T={T} p_min={pmin}", rows, T, pmin, got, seeds, 0, 0)


def test_minp_all_rows_one_point(rgd, z):
    seeds = np.arange(256, dtype=np.uint64)
    got = sample_gpu(rgd, z, 2.0, 0.05, seeds, ctr=7, stream0=0)[:, 0]
    _check_rows("sampler sweep, 256 rows, T=2 p_min=0.05", z, 2.0, 0.05, got, seeds, 7, 0)


def test_thousand_draws_match_and_follow_kept_distribution(rgd, z):
    from scipy import stats
    rows = z[:6]
    seeds = np.arange(6, dtype=np.uint64) + 1000
    T, pmin, D = 1.5, 0.1, 1000
    got = sample_gpu(rgd, rows, T, pmin, seeds, ctr=0, stream0=0, draws=D)
    for r in range(rows.shape[0]):
        us = philox.uniform(int(seeds[r]), 0, np.arange(D, dtype=np.uint64))
        draws = sampler.sample_minp_many(rows[r], T, pmin, us)
        ok = np.array([d.cdf_margin >= MARGIN and d.logit_margin >= MARGIN for d in draws])
        want = np.array([d.token for d in draws])
        assert np.array_equal(got[r][ok], want[ok])
        for i in np.flatnonzero(~ok):
            judge_draw(rows[r], T, pmin, float(us[i]), int(got[r][i]))
        p = sampler.kept_probabilities(rows[r], T, pmin)
        support = np.flatnonzero(p > 0)
        assert set(np.unique(got[r])) <= set(support)
        exp = p[support] * D
        obs = np.bincount(got[r], minlength=len(p))[support]
        big = exp >= 5
        o = np.append(obs[big], obs[~big].sum())
        e = np.append(exp[big], exp[~big].sum())
        if e[-1] < 1e-9:
            o, e = o[:-1], e[:-1]
        if len(e) > 1:
            assert stats.chisquare(o, e).pvalue > 1e-4


def test_edge_cases_tiny_vocab(rgd):
    z = np.array([[0.0, 3.0, 1.0, 3.0, -2.0, 0.5, 2.9, 1.0]] * 4, np.float32)
    seeds = np.arange(4, dtype=np.uint64)
    got = sample_gpu(rgd, z, 1.0, 1.0, seeds, draws=50)
    assert set(np.unique(got)) == {1, 3}   # p_min = 1 keeps exactly the tied maxima
    got = sample_gpu(rgd, z, 1.0, 0.0, seeds, draws=400)
    assert set(np.unique(got)) == set(range(8))
    got = sample_gpu(rgd, z, 5.0, 0.5, seeds, draws=200)
    kept = sampler.minp_weights(z[0], 5.0, 0.5)[1]
    assert set(np.unique(got)) <= set(np.flatnonzero(kept))


def test_deterministic(rgd, z):
    seeds = np.arange(64, dtype=np.uint64) * 7919
    a = sample_gpu(rgd, z[:64], 3.0, 0.05, seeds, ctr=3, draws=4)
    b = sample_gpu(rgd, z[:64], 3.0, 0.05, seeds, ctr=3, draws=4)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("T,pmin", [(0.7, 0.05), (2.0, 0.05), (3.0, 0.05), (3.0, 0.2)])
def test_minp_one_workgroup_per_row_with_further_draws(rgd, z, T, pmin):
    """128 or more rows take the one-launch path (one workgroup per row, which
    also settles the chunk sums that later draws reuse); 3 draws per row, from
    no window chunk at all (T = 0.7) to every chunk inside the window (T = 3,
    p_min = 0.05)."""
    rows = z[:160]
    seeds = np.arange(160, dtype=np.uint64) * 31 + 5
    D = 3
    got = sample_gpu(rgd, rows, T, pmin, seeds, ctr=11, stream0=2, draws=D)
    tally = Tally(f"sampler sweep, 160 rows x 3 draws (row kernel), T={T} p_min={pmin}")
    for r in range(rows.shape[0]):
        for d in range(D):
            u = float(philox.uniform(int(seeds[r]), 11, 2 + d))
            tally.add(judge_draw(rows[r], T, pmin, u, int(got[r, d])))
    tally.close()


def test_edge_cases_tiny_vocab_many_rows(rgd):
    z = np.array([[0.0, 3.0, 1.0, 3.0, -2.0, 0.5, 2.9, 1.0]] * 130, np.float32)
    seeds = np.arange(130, dtype=np.uint64)
    got = sample_gpu(rgd, z, 1.0, 1.0, seeds, draws=4)
    assert set(np.unique(got)) == {1, 3}
    got = sample_gpu(rgd, z, 1.0, 0.0, seeds, draws=8)
    assert set(np.unique(got)) == set(range(8))


@pytest.mark.parametrize("R", [1, 130])
@pytest.mark.parametrize("V", [4100, 12288 + 4])
def test_minp_ragged_last_chunk(rgd, R, V):
    """A last 4096-logit chunk holding 4 logits, through the chunk kernels (1
    row) and the one-workgroup-per-row kernel (130 rows): the maximum and a
    heavy token placed in the ragged chunk."""
    g = np.random.default_rng(V + R)
    z = g.normal(size=(R, V)).astype(np.float32)
    z[:, V - 2] = 6.0            # the row maximum, in the ragged last chunk
    z[::2, V - 3] = 5.5
    seeds = np.arange(R, dtype=np.uint64) + 3
    for T, pmin in ((1.0, 0.1), (3.0, 0.05)):
        got = sample_gpu(rgd, z, T, pmin, seeds, ctr=1, stream0=0, draws=2)
        for r in range(R):
            for d in range(2):
                judge_draw(z[r], T, pmin, float(philox.uniform(int(seeds[r]), 1, d)), int(got[r, d]))
