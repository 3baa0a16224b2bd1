"""p-less sampling on the GPU vs the oracle (the truncation rule of the cited
p-less paper, temperature first: keep p_i >= sum_j p_j^2): the standalone
kernel on the sampler-sweep logits (every temperature, all 256 rows, 1000 draws
per row with a chi-square test), small hand-checked rows, and the decode path
of the tiny fp32 decoder, free-running and teacher-forced."""
import numpy as np
import pytest

import synth
from oracle import philox, pless
from oracle import rgd as orgd
from oracle.model import Decoder, KVCache
from tests.gpu_common import Tally, judge_draw_pless, rel_err, seeds_tensor, torch

pytestmark = pytest.mark.gpu
MARGIN = 1e-4
W0 = synth.TINY_FP32


@pytest.fixture(scope="module")
def rgd():
    import paper_2607_20791_amd as m
    return m


@pytest.fixture(scope="module")
def z():
    return synth.sweep_logits()


def sample_pless_gpu(rgd, z_np, T, seeds, ctr=0, stream0=0, draws=1):
    t = torch()
    z = t.from_numpy(np.ascontiguousarray(z_np, dtype=np.float32)).cuda()
    R, V = z.shape
    ws = t.empty(rgd.sampler_workspace_bytes(R, V), dtype=t.uint8, device="cuda")
    out = t.full((R, draws), -1, dtype=t.int32, device="cuda")
    rgd.kernel_sample_pless(z, T, seeds_tensor(seeds), ctr, stream0, draws, ws, out)
    t.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("T", synth.SWEEP.temperatures)
def test_pless_single_draw_every_temperature(rgd, z, T):
    rows = z[:48]
    seeds = np.arange(48, dtype=np.uint64) + 500
    got = sample_pless_gpu(rgd, rows, T, seeds, ctr=3)[:, 0]
    tally = Tally(f"p-less, sampler sweep, 48 rows, T={T}")
    for r in range(48):
        tally.add(judge_draw_pless(rows[r], T, float(philox.uniform(int(seeds[r]), 3, 0)), int(got[r])))
    # every draw was judged above (exact outside margin cases); from T = 2 on the
    # threshold falls inside the dense N(0, 1) tail, so most rows are margin
    # cases, nearly all of which still give the oracle's token
    tally.close()


def test_pless_all_rows_and_further_draws(rgd, z):
    seeds = np.arange(256, dtype=np.uint64) * 7 + 1
    got = sample_pless_gpu(rgd, z, 2.0, seeds, ctr=9, stream0=4, draws=2)
    tally = Tally("p-less, sampler sweep, 256 rows x 2 draws, T=2")
    for r in range(256):
        for d in range(2):
            u = float(philox.uniform(int(seeds[r]), 9, 4 + d))
            tally.add(judge_draw_pless(z[r], 2.0, u, int(got[r, d])))
    tally.close()


def test_pless_thousand_draws_follow_the_kept_distribution(rgd, z):
    from scipy import stats
    rows = z[:4]
    seeds = np.arange(4, dtype=np.uint64) + 2000
    T, D = 3.0, 1000
    got = sample_pless_gpu(rgd, rows, T, seeds, draws=D)
    for r in range(4):
        us = philox.uniform(int(seeds[r]), 0, np.arange(D, dtype=np.uint64))
        draws = pless.sample_pless_many(rows[r], T, us)
        ok = np.array([d.cdf_margin >= MARGIN and d.logit_margin >= MARGIN for d in draws])
        assert np.array_equal(got[r][ok], np.array([d.token for d in draws])[ok])
        q = pless.kept_probabilities(rows[r], T)
        support = np.flatnonzero(q > 0)
        assert set(np.unique(got[r])) <= set(support)
        exp = q[support] * D
        obs = np.bincount(got[r], minlength=len(q))[support]
        big = exp >= 5
        o = np.append(obs[big], obs[~big].sum())
        e = np.append(exp[big], exp[~big].sum())
        if e[-1] < 1e-9:
            o, e = o[:-1], e[:-1]
        if len(e) > 1:
            assert stats.chisquare(o, e).pvalue > 1e-4


def test_pless_hand_checked_rows(rgd):
    pad = -1e4
    rows = np.array([
        [1.5] * 8,                                                        # uniform: all kept
        np.log([0.1, 0.3, 0.2, 0.3, 0.1, 1e-30, 1e-30, 1e-30]).tolist(),  # sum p^2 = 0.24: 1 and 3
        [0.0, 2.0, pad, pad, pad, pad, pad, pad],                          # two tokens: the larger
        np.log([0.35, 0.25, 0.2, 0.1, 0.1, 1e-30, 1e-30, 1e-30]).tolist(),  # 0.245: 0 and 1
    ], np.float32)
    rows[3] *= 2.0                       # at T = 2 row 3 is p = (0.35, 0.25, 0.2, 0.1, 0.1) again
    seeds = np.arange(4, dtype=np.uint64)
    got1 = sample_pless_gpu(rgd, rows[:3], 1.0, seeds[:3], draws=400)
    assert set(np.unique(got1[0])) == set(range(8))
    assert set(np.unique(got1[1])) == {1, 3}
    assert set(np.unique(got1[2])) == {1}
    got2 = sample_pless_gpu(rgd, rows[3:], 2.0, seeds[3:], draws=400)
    assert set(np.unique(got2[0])) == {0, 1}


@pytest.fixture(scope="module")
def tiny():
    weights = synth.model_weights(W0)
    dec = Decoder(weights)
    prompts = synth.prompt_tokens(W0)
    caches, last = [], []
    for b in range(W0.n_prompts):
        c = KVCache(W0.n_layers)
        last.append(dec.prefill(prompts[b], c))
        caches.append(c)
    return dict(weights=weights, dec=dec, prompts=prompts, caches=caches, last=last)


def _tiny_gpu(rgd, tiny):
    from paper_2607_20791_amd import session
    t = torch()
    m = session.build_model(tiny["weights"], max_rows=64, max_pos=128)
    kv = session.alloc_kv(m, W0, max_prompts=W0.n_prompts, max_prefix=W0.prompt_len, n_pages=96)
    last = t.empty(W0.n_prompts, W0.vocab, dtype=t.float32, device="cuda")
    rgd.prefill_kv(m, kv, session.to_device(tiny["prompts"]), 0, last)
    return m, kv, last


def test_pless_decode_path_free_running(rgd, tiny):
    t = torch()
    m, kv, last = _tiny_gpu(rgd, tiny)
    prompts, N, S, T = [0, 3, 6, 9], 2, 24, 2.0
    seeds = np.arange(len(prompts) * N, dtype=np.uint64) + 40
    out = t.full((len(prompts), N, S), -1, dtype=t.int32, device="cuda")
    rgd.sample_continuations_pless(m, kv, last, prompts, N, S, T, seeds_tensor(seeds), out)
    t.cuda.synchronize()
    rgd.check_status(m)
    got = out.cpu().numpy().reshape(-1, S)
    tally = Tally("p-less, tiny fp32 decoder free-running, 8 branches x 24 tokens")
    for r in range(len(prompts) * N):
        b = prompts[r // N]
        br = orgd.sample_branch(tiny["dec"], tiny["caches"][b], tiny["last"][b], int(seeds[r]), S, T, 0.0,
                                keep_logits=True, truncation="pless")
        for s in range(S):
            v = tally.add(judge_draw_pless(br.logits[s], T, float(philox.uniform(int(seeds[r]), s)),
                                           int(got[r, s])))
            if v == "margin-diff":
                break       # the histories differ from here on
    # a branch is compared draw by draw until its first margin-diff draw (its
    # history then differs from the oracle's); at most one branch may diverge
    tally.close(max_diff_frac=0.0)
    # deterministic: the same call gives the same tokens
    out2 = t.full_like(out, -1)
    rgd.sample_continuations_pless(m, kv, last, prompts, N, S, T, seeds_tensor(seeds), out2)
    t.cuda.synchronize()
    assert t.equal(out, out2)


def test_pless_decode_path_teacher_forced(rgd, tiny):
    """Per-step logits of forced histories match the oracle at 1e-5 and each
    drawn token is the oracle's p-less draw on them (margin rule)."""
    t = torch()
    from paper_2607_20791_amd import session
    m, kv, last = _tiny_gpu(rgd, tiny)
    prompts, N, S, T = [2, 7], 2, 10, 1.5
    forced = synth.forced_history(W0, len(prompts) * N, S)
    seeds = np.arange(len(prompts) * N, dtype=np.uint64) + 91
    out = t.full((len(prompts), N, S), -1, dtype=t.int32, device="cuda")
    tap = t.empty(S, len(prompts) * N, W0.vocab, dtype=t.float32, device="cuda")
    rgd.sample_continuations_pless(m, kv, last, prompts, N, S, T, seeds_tensor(seeds), out,
                                   forced=session.to_device(forced), logits_tap=tap)
    t.cuda.synchronize()
    tap_h, got = tap.cpu().numpy(), out.cpu().numpy().reshape(-1, S)
    for r in range(len(prompts) * N):
        b = prompts[r // N]
        br = orgd.sample_branch(tiny["dec"], tiny["caches"][b], tiny["last"][b], int(seeds[r]), S, T, 0.0,
                                forced=forced[r], keep_logits=True, truncation="pless")
        assert rel_err(tap_h[:, r], np.stack(br.logits)).max() <= 1e-5
        for s in range(S):
            judge_draw_pless(br.logits[s], T, float(philox.uniform(int(seeds[r]), s)), int(got[r, s]))


@pytest.mark.parametrize("V", [8, 4100])
def test_pless_ragged_and_tiny_vocabularies(rgd, V):
    g = np.random.default_rng(V)
    z = g.normal(size=(5, V)).astype(np.float32) * 2
    z[1, V - 1] = 9.0
    seeds = np.arange(5, dtype=np.uint64) + 7
    for T in (0.7, 2.0):
        got = sample_pless_gpu(rgd, z, T, seeds, ctr=2, draws=3)
        for r in range(5):
            for d in range(3):
                judge_draw_pless(z[r], T, float(philox.uniform(int(seeds[r]), 2, d)), int(got[r, d]))
