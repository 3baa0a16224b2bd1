"""The bf16 8B-shaped decode layer end to end, at the 512- and 8192-position
synthetic prefixes (1 layer, d=4096, 32/8 heads, ffn 14336, V=128256).

Oracle parity on sampled outputs: the last-position logits of the prompt and
the logits of teacher-forced branches at their first steps, within the bf16
tolerance; every draw is checked against the oracle sampler on the logits the
GPU computed (tapped in fp32).  Properties at the full sizes of the benchmark
(P=8192, N=64, 128 steps): runs are bit-deterministic, the shared prompt KV is
never modified, and a gated miss samples exactly what ungated sampling does."""
import numpy as np
import pytest

import synth
from oracle import philox
from oracle import rgd as orgd
from oracle.model import Decoder, KVCache
from tests.gpu_common import Tally, judge_draw, judge_draw_pless, rel_err, seeds_tensor, torch

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module")
def rgd():
    import paper_2607_20791_amd as m
    return m


class World:
    """One 8B-shaped layer over a synthetic prefix: device model and KV state
    (row capacity max_rows) and the oracle decoder with the prompt's logits."""

    def __init__(self, rgd, w, max_rows=64, weights=None):
        from paper_2607_20791_amd import session
        t = torch()
        self.w = w
        self.weights = synth.model_weights(w) if weights is None else weights
        self.P = w.synthetic_prefix
        self.kp, self.vp = synth.synthetic_prefix_kv(w, 0)
        self.last_tok = int(synth.prompt_tokens(w)[0, 0])
        self.model = session.build_model(self.weights, max_rows=max_rows, max_pos=self.P + 256)
        self.kv = session.alloc_kv(self.model, w, max_prompts=1, max_prefix=self.P + 1,
                                   n_pages=max_rows * 8 + 24)
        session.fill_prefix(self.kv, 0, self.kp, self.vp)
        self.last = t.empty(1, w.vocab, dtype=t.float32, device="cuda")
        self.tok = t.tensor([[self.last_tok]], dtype=t.int32, device="cuda")
        self.dec = Decoder(self.weights)
        self.cache = KVCache.from_arrays([self.kp[0]], [self.vp[0]])
        self.ref_last = self.dec.prefill([self.last_tok], self.cache, start_pos=self.P)

    def prefill(self, rgd):
        self.kv.set_prefix_len(0, self.P)
        rgd.prefill_kv(self.model, self.kv, self.tok, self.P, self.last)


@pytest.fixture(scope="module")
def p512(rgd):
    return World(rgd, synth.LAYER_P512)


@pytest.fixture(scope="module")
def p8192(rgd):
    return World(rgd, synth.LAYER_P8192)


def _last_logits(rgd, wd):
    t = torch()
    wd.prefill(rgd)
    t.cuda.synchronize()
    err = rel_err(wd.last.cpu().numpy()[0], wd.ref_last)
    print(wd.w.name, "last-position logits rel err", err)
    assert err <= TOL


def _teacher_forced(rgd, wd, rows, steps, T, p_min, pless=False):
    t = torch()
    from paper_2607_20791_amd import session
    wd.prefill(rgd)
    w, V = wd.w, wd.w.vocab
    forced = synth.forced_history(w, rows, steps)
    seeds = synth.branch_seeds(1, rows, base=500)
    out = t.full((1, rows, steps), -1, dtype=t.int32, device="cuda")
    tap = t.empty(steps, rows, V, dtype=t.float32, device="cuda")
    if pless:
        rgd.sample_continuations_pless(wd.model, wd.kv, wd.last, [0], rows, steps, T, seeds_tensor(seeds), out,
                                       forced=session.to_device(forced), logits_tap=tap)
    else:
        rgd.sample_continuations(wd.model, wd.kv, wd.last, [0], rows, steps, T, p_min, seeds_tensor(seeds), out,
                                 forced=session.to_device(forced), logits_tap=tap)
    t.cuda.synchronize()
    rgd.check_status(wd.model)
    tap_h, got = tap.cpu().numpy(), out.cpu().numpy()[0]
    worst = 0.0
    tally = Tally(f"{w.name} teacher-forced{' p-less' if pless else ''}, {rows} rows x {steps} tokens")
    for r in range(rows):
        br = orgd.sample_branch(wd.dec, wd.cache, wd.ref_last, int(seeds[r]), steps, T, p_min,
                                forced=forced[r], keep_logits=True, truncation="pless" if pless else "minp")
        err = rel_err(tap_h[:, r], np.stack(br.logits))
        worst = max(worst, float(err.max()))
        assert err.max() <= TOL, (r, err)
        for s in range(steps):   # the sampler on the GPU's own logits
            u = float(philox.uniform(int(seeds[r]), s))
            if pless:
                tally.add(judge_draw_pless(tap_h[s, r], T, u, int(got[r, s])))
            else:
                tally.add(judge_draw(tap_h[s, r], T, p_min, u, int(got[r, s])))
    print(w.name, "teacher-forced logits rel err (worst)", worst)
    tally.close()


def test_bf16_p512_prompt_logits(rgd, p512):
    _last_logits(rgd, p512)


def test_bf16_p512_teacher_forced(rgd, p512):
    _teacher_forced(rgd, p512, rows=2, steps=3, T=p512.w.temperature, p_min=p512.w.min_p)


def test_bf16_p512_teacher_forced_pless(rgd, p512):
    """p-less truncation on the 8B-shaped layer: logits within the bf16
    tolerance and each token the oracle's p-less draw on the GPU's logits."""
    _teacher_forced(rgd, p512, rows=2, steps=3, T=p512.w.temperature, p_min=0.0, pless=True)


def test_bf16_p8192_prompt_logits(rgd, p8192):
    _last_logits(rgd, p8192)


def test_bf16_p8192_teacher_forced(rgd, p8192):
    _teacher_forced(rgd, p8192, rows=2, steps=2, T=p8192.w.temperature, p_min=p8192.w.min_p)


def test_bf16_p8192_full_size_properties(rgd, p8192):
    """N=64 branches x 128 steps from the 8192-position prefix: deterministic,
    prefix untouched, and a gated miss (typical 0%-hit table) equals ungated."""
    t = torch()
    w = p8192.w
    N, S, k = w.n_branches, w.steps, w.probe_k
    seeds = seeds_tensor(synth.branch_seeds(1, N))
    before = (p8192.kv.prefix_k.clone(), p8192.kv.prefix_v.clone())

    def ungated():
        p8192.prefill(rgd)
        out = t.full((1, N, S), -1, dtype=t.int32, device="cuda")
        rgd.sample_continuations(p8192.model, p8192.kv, p8192.last, [0], N, S, w.temperature, w.min_p, seeds, out)
        t.cuda.synchronize()
        rgd.check_status(p8192.model)
        return out

    a, b = ungated(), ungated()
    assert t.equal(a, b)
    assert int(a.min()) >= 0 and int(a.max()) < w.vocab
    # gated: probe against the typical table, then the miss is sampled
    off, toks = synth.random_table(w)
    table = rgd.Table(off, toks)
    p8192.prefill(rgd)
    ptok = t.empty(1, k, dtype=t.int32, device="cuda")
    plen = t.empty(1, dtype=t.int32, device="cuda")
    ev = t.empty(1, dtype=t.int32, device="cuda")
    rgd.probe(p8192.model, p8192.kv, p8192.last, table, 1, k, 3, -1, ptok, plen, ev)
    dec, miss = rgd.gate(p8192.kv, ev, 1)
    assert dec[0] == 0 and list(miss) == [0]
    out = t.full((1, N, S), -1, dtype=t.int32, device="cuda")
    rgd.sample_continuations(p8192.model, p8192.kv, p8192.last, list(miss), N, S, w.temperature, w.min_p, seeds, out)
    t.cuda.synchronize()
    assert t.equal(out, a)
    assert t.equal(before[0], p8192.kv.prefix_k) and t.equal(before[1], p8192.kv.prefix_v)
    # the probe's first token is the argmax of the prompt's last logits
    assert int(ptok[0, 0]) == int(p8192.last[0].argmax())


@pytest.mark.parametrize("layer", [0, 1])
def test_p512_residual_precheck_score(rgd, p512, layer):
    """Residual-stream classifier pre-check (Appendix A) on the 8B-shaped layer:
    the score of the prefilled last token within the bf16 tolerance of the
    oracle's, and the prefill's logits unchanged by the readout."""
    t = torch()
    d = p512.w.d_model
    g = np.random.default_rng(11 + layer)
    w = (g.normal(size=d) / np.sqrt(d)).astype(np.float32)
    b = 0.1
    scores = t.empty(1, dtype=t.float32, device="cuda")
    plain = p512.last.clone()
    p512.prefill(rgd)
    plain.copy_(p512.last)
    p512.kv.set_prefix_len(0, p512.P)
    rgd.prefill_kv_scored(p512.model, p512.kv, p512.tok, p512.P, p512.last, layer, t.from_numpy(w).cuda(), b, scores)
    t.cuda.synchronize()
    assert t.equal(plain, p512.last)
    taps = {}
    cache = KVCache.from_arrays([p512.kp[0]], [p512.vp[0]])
    p512.dec.prefill([p512.last_tok], cache, start_pos=p512.P, taps=taps)
    from oracle import precheck
    ref = precheck.residual_score(taps[layer], w.astype(np.float64), b)
    got = float(scores.item())
    print("512-prefix layer: pre-check score after block", layer, got, "oracle", ref)
    assert abs(got - ref) <= TOL
