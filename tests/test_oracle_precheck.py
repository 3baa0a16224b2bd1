"""Pins for the residual-stream classifier pre-check and the adaptive gate
(Appendix A; not GPU): the logistic readout against closed forms, the residual
taps against the model's own logits and block, and the adaptive decision's
limits (theta below every score: the plain gate; theta at 1: direct sampling)."""
import numpy as np
import pytest

import synth
from oracle import gate, precheck, rgd, sampler
from oracle.model import Decoder, KVCache, rmsnorm, linear

TINY = synth.scaled(synth.TINY_FP32, name="tiny-pre", n_layers=2, d_model=32, n_heads=4, n_kv_heads=2,
                    head_dim=8, ffn=48, vocab=61, weight_std=0.5)
PROMPT = [3, 14, 15, 9, 2, 6]


def test_logistic_readout_closed_forms():
    h = np.array([1.0, 2.0])
    assert precheck.residual_score(h, [0.5, -0.25], 0.0) == 0.5              # w . h = 0
    assert np.isclose(precheck.residual_score(h, [0.5, -0.25], np.log(3.0)), 0.75)   # 3 / (1 + 3)
    assert np.isclose(precheck.residual_score(h, [0.0, 0.0], -np.log(4.0)), 0.2)     # w = 0: sigmoid(b)
    assert np.isclose(precheck.residual_score(h, [1.0, 1.0], 0.0), 1 / (1 + np.exp(-3.0)))
    z = np.linspace(-5, 5, 11)
    p = [precheck.residual_score([1.0], [x], 0.0) for x in z]
    assert all(a < b for a, b in zip(p, p[1:]))                              # monotone in w . h


def test_taps_are_the_residual_stream():
    dec = Decoder(synth.model_weights(TINY))
    taps = {}
    last = dec.prefill(PROMPT, KVCache(TINY.n_layers), taps=taps)
    assert sorted(taps) == [0, 1, 2]
    # layer 0 is the embedding of the last prompt token
    assert np.array_equal(taps[0], dec.embed([PROMPT[-1]])[0])
    # the last layer's residual is what the final norm and LM head read
    W = dec.W
    assert np.allclose(linear(W.lm_head, rmsnorm(taps[2], W.final_norm, TINY.rms_eps)), last)
    # a one-block model tapped at block 1 sees the same residual as block 1 of the two-block one
    one = Decoder(synth.Weights(synth.scaled(TINY, n_layers=1), W.embed, W.final_norm, W.lm_head,
                                W.layers[:1]))
    t1 = {}
    one.prefill(PROMPT, KVCache(1), taps=t1)
    assert np.allclose(t1[1], taps[1])


@pytest.mark.parametrize("soft", [None, (3, 4, 0.01)])
def test_adaptive_gate_limits(soft):
    dec = Decoder(synth.model_weights(TINY))
    g = np.random.default_rng(5)
    w = g.normal(size=TINY.d_model) / np.sqrt(TINY.d_model)
    table = [[7, 8, 9]]
    seeds = [4, 5]
    # theta = 0: no score is <= 0, so the gate of Algorithm 1 decides as without the pre-check
    r0 = precheck.adaptive_gated(dec, PROMPT, table, 6, seeds, 4, 2.0, 0.1, 2, w, 0.3, 0.0, soft=soft)
    assert not r0.skipped and 0.0 < r0.score < 1.0
    prefix = KVCache(TINY.n_layers)
    last = dec.prefill(PROMPT, prefix)
    if soft is None:
        plain = rgd.refusal_gated(dec, None, table, 6, seeds, 4, 2.0, 0.1, prefix=prefix, last_logits=last)
        assert (r0.gated.hit, r0.gated.probe, r0.gated.event) == (plain.hit, plain.probe, plain.event)
    # theta = 1: every prompt skips the check; its branches are the ungated samples
    r1 = precheck.adaptive_gated(dec, PROMPT, table, 6, seeds, 4, 2.0, 0.1, 2, w, 0.3, 1.0, soft=soft)
    assert r1.skipped and r1.gated.probe == [] and not r1.gated.hit
    for s, br in zip(seeds, r1.gated.branches):
        assert br.tokens == rgd.sample_branch(dec, prefix, last, s, 4, 2.0, 0.1).tokens
    # the decision is P <= theta, at the score itself
    r2 = precheck.adaptive_gated(dec, PROMPT, table, 6, seeds, 4, 2.0, 0.1, 2, w, 0.3, r0.score, soft=soft)
    assert r2.skipped


def test_score_reads_the_residual_after_the_chosen_block():
    """The pre-check scores the residual after block `layer` (0: the embedding):
    each layer's score equals the readout of that tap, and the taps differ."""
    dec = Decoder(synth.model_weights(TINY))
    taps = {}
    dec.prefill(PROMPT, KVCache(TINY.n_layers), taps=taps)
    w = np.random.default_rng(8).normal(size=TINY.d_model)
    scores = []
    for layer in range(TINY.n_layers + 1):
        r = precheck.adaptive_gated(dec, PROMPT, [[7, 8]], 4, [1], 2, 2.0, 0.1, layer, w, 0.1, 1.0)
        assert r.score == precheck.residual_score(taps[layer], w, 0.1)
        scores.append(r.score)
    assert len(set(scores)) == len(scores)
