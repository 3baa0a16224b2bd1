"""Algorithm 1 end to end on the oracle (not GPU): a hit returns the greedy
probe, a miss returns exactly the ungated sampling output (distribution
preservation, Section 2/3), and branches never see probe tokens."""
import numpy as np

import synth
from oracle import gate, philox, rgd, sampler
from oracle.model import Decoder, KVCache

TINY = synth.scaled(synth.TINY_FP32, name="tiny-rgd", n_layers=1, d_model=32, n_heads=4, n_kv_heads=2,
                    head_dim=8, ffn=48, vocab=61, weight_std=0.5)


def _setup():
    dec = Decoder(synth.model_weights(TINY))
    prefix = KVCache(1)
    last = dec.prefill([3, 14, 15, 9, 2], prefix)
    return dec, prefix, last


def test_hit_returns_greedy_probe():
    dec, prefix, last = _setup()
    q_free, _ = rgd.greedy_probe(dec, prefix, last, table=[], k=6)    # only token 1
    # build a table whose entry is the model's own first greedy tokens
    q6, ev = rgd.greedy_probe(dec, prefix, last, table=[[q_free[0], -1]], k=6)
    assert ev == gate.INCOMPAT and len(q6) == 2
    full = [q_free[0]]
    tail = KVCache(1)
    for _ in range(5):
        full.append(sampler.argmax(dec.decode(full[-1], prefix, tail)))
    res = rgd.refusal_gated(dec, None, [full[:3]], 6, seeds=[1, 2], steps=4, T=2.0, p_min=0.1,
                            prefix=prefix, last_logits=last)
    assert res.hit and res.probe == full and res.event == gate.MAXLEN and res.branches == []


def test_miss_equals_ungated_sampling():
    dec, prefix, last = _setup()
    seeds = [11, 12, 13]
    res = rgd.refusal_gated(dec, None, [[-5, -6]], 6, seeds=seeds, steps=5, T=2.0, p_min=0.1,
                            prefix=prefix, last_logits=last)
    assert not res.hit and res.event == gate.INCOMPAT
    for s, br in zip(seeds, res.branches):
        ung = rgd.sample_branch(dec, prefix, last, s, 5, 2.0, 0.1)
        assert br.tokens == ung.tokens
    # the prefix cache was not changed by the probe or the branches
    assert prefix.length() == 5


def test_branch_first_token_uses_prompt_logits_and_counter_zero():
    dec, prefix, last = _setup()
    br = rgd.sample_branch(dec, prefix, last, 77, 3, 1.5, 0.05)
    u0 = float(philox.uniform(77, 0))
    assert br.tokens[0] == sampler.sample_minp(last, 1.5, 0.05, u0).token


def test_branch_step_s_draws_with_counter_s_and_its_stream():
    """Token s of a branch uses the uniform of Philox counter (s, stream, 0, 0)
    under key (seed lo, seed hi), formed here from the scalar Philox that the
    known-answer vectors pin; the whole draw (token and margins) must match."""
    dec, prefix, last = _setup()
    seed = (5 << 32) | 77
    for stream in (0, 3):
        br = rgd.sample_branch(dec, prefix, last, seed, 5, 1.5, 0.05, keep_logits=True, stream=stream)
        for s in range(5):
            w0 = philox.philox4x32_10_int((s, stream, 0, 0), (seed & 0xFFFFFFFF, seed >> 32))[0]
            u = (w0 >> 8) * 2.0 ** -24
            assert br.draws[s] == sampler.sample_minp(br.logits[s], 1.5, 0.05, u)


def test_probe_ending_on_the_stop_token_is_a_hit():
    """A compatible probe that emits the stop token ends the gate with STOP, and
    Algorithm 1 returns the greedy probe (no branches)."""
    dec, prefix, last = _setup()
    full = [sampler.argmax(last)]
    tail = KVCache(1)
    for _ in range(3):
        full.append(sampler.argmax(dec.decode(full[-1], prefix, tail)))
    eos = full[1]
    stop_at = full.index(eos) + 1
    res = rgd.refusal_gated(dec, None, [full], 6, seeds=[1, 2], steps=4, T=2.0, p_min=0.1, eos=eos,
                            prefix=prefix, last_logits=last)
    assert res.event == gate.STOP and res.hit and res.probe == full[:stop_at] and res.branches == []


def test_forced_history_changes_only_inputs():
    dec, prefix, last = _setup()
    forced = [4, 8, 15, 16]
    a = rgd.sample_branch(dec, prefix, last, 5, 5, 2.0, 0.1, forced=forced, keep_logits=True)
    # logits at step s are those of the forced history
    tail = KVCache(1)
    for s in range(4):
        want = dec.decode(forced[s], prefix, tail)
        assert np.allclose(a.logits[s + 1], want)
