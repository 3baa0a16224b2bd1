"""Pins for the oracle decoder (not GPU): closed forms, brute force, and
decode-versus-prefill consistency."""
import math

import numpy as np
import pytest

import synth
from oracle import model as om
from oracle.model import Decoder, KVCache

TINY = synth.scaled(synth.TINY_FP32, name="tiny", n_layers=2, d_model=32, n_heads=4, n_kv_heads=2,
                    head_dim=8, ffn=48, vocab=97, weight_std=0.3)


def test_rope_closed_form_d4():
    theta = 10000.0
    for pos in (0, 1, 5):
        x = np.array([[1.0, 0.0, 0.0, 0.0], [0.0, 1.0, 0.0, 0.0]])
        y = om.rope(x, pos, theta)
        a0, a1 = pos * 1.0, pos * theta ** -0.5
        assert np.allclose(y[0], [math.cos(a0), 0, math.sin(a0), 0])
        assert np.allclose(y[1], [0, math.cos(a1), 0, math.sin(a1)])
        x3 = np.array([[0.0, 0.0, 1.0, 0.0]])
        assert np.allclose(om.rope(x3, pos, theta)[0], [-math.sin(a0), 0, math.cos(a0), 0])


def test_rope_norm_and_relative_position():
    g = np.random.default_rng(0)
    q, k = g.normal(size=(2, 1, 64))
    assert np.allclose(np.linalg.norm(om.rope(q, 37, 5e5)), np.linalg.norm(q))
    d1 = om.rope(q, 10, 5e5)[0] @ om.rope(k, 3, 5e5)[0]
    d2 = om.rope(q, 107, 5e5)[0] @ om.rope(k, 100, 5e5)[0]
    assert np.isclose(d1, d2)


def test_rmsnorm_and_silu_closed_forms():
    x = np.array([3.0, -4.0])                       # mean square 12.5
    assert np.allclose(om.rmsnorm(x, np.ones(2), 0.0), x / math.sqrt(12.5))
    assert np.allclose(om.rmsnorm(x, np.array([2.0, 0.5]), 0.0), x / math.sqrt(12.5) * [2, .5])
    assert om.silu(np.array([0.0]))[0] == 0.0
    assert np.isclose(om.silu(np.array([1.0]))[0], 1.0 / (1.0 + math.exp(-1.0)))


def test_linear_matches_loops_and_widening_is_exact():
    g = np.random.default_rng(1)
    w32 = g.normal(size=(5, 7)).astype(np.float32)
    x = g.normal(size=7)
    want = [sum(float(w32[o, i]) * x[i] for i in range(7)) for o in range(5)]
    assert np.allclose(om.linear(w32, x, chunk_rows=2), want, rtol=1e-13)
    bits = synth.to_bf16_bits(w32)
    assert np.array_equal(om.widen(bits), synth.bf16_bits_to_f32(bits).astype(np.float64))
    assert om.widen(np.array([0x3F80], np.uint16))[0] == 1.0
    assert om.widen(np.array([0xC040], np.uint16))[0] == -3.0


@pytest.fixture(scope="module")
def tiny():
    return Decoder(synth.model_weights(TINY))


def test_decode_matches_prefill(tiny):
    toks = np.array([5, 17, 3, 88, 41, 2, 60])
    full = KVCache(TINY.n_layers)
    want = tiny.prefill(toks, full)
    # prefill a prefix, then decode the rest one token at a time
    pre = KVCache(TINY.n_layers)
    tiny.prefill(toks[:4], pre)
    tail = KVCache(TINY.n_layers)
    for t in toks[4:]:
        got = tiny.decode(int(t), pre, tail)
    assert np.allclose(got, want, rtol=1e-11, atol=1e-11)
    # the cache rows written by prefill equal those appended by decode
    for l in range(TINY.n_layers):
        assert np.allclose(np.array(pre.k[l] + tail.k[l]), np.array(full.k[l]))


def test_prefill_in_two_segments(tiny):
    toks = np.array([1, 2, 3, 4, 5, 6])
    a = KVCache(TINY.n_layers)
    la = tiny.prefill(toks, a)
    b = KVCache(TINY.n_layers)
    tiny.prefill(toks[:2], b)
    lb = tiny.prefill(toks[2:], b, start_pos=2)
    assert np.allclose(la, lb, rtol=1e-11, atol=1e-11)


def test_first_token_brute_force(tiny):
    """A one-token prompt attends only to itself: the block reduces to
    x + Wo (v replicated per group) + FFN, computed here by hand."""
    W = tiny.W
    L = W.layers[0]
    x = om.widen(W.embed[7])
    a = x / math.sqrt(np.mean(x * x) + TINY.rms_eps)
    v = om.widen(L["wv"]) @ a
    G = TINY.n_heads // TINY.n_kv_heads
    o = np.concatenate([v[(h // G) * 8:(h // G + 1) * 8] for h in range(TINY.n_heads)])
    h = x + om.widen(L["wo"]) @ o
    b = h / math.sqrt(np.mean(h * h) + TINY.rms_eps)
    gt = om.widen(L["w_gate"]) @ b
    f = gt / (1 + np.exp(-gt)) * (om.widen(L["w_up"]) @ b)
    x1 = h + om.widen(L["w_down"]) @ f
    one_layer = synth.scaled(TINY, n_layers=1)
    dec = Decoder(synth.Weights(one_layer, W.embed, W.final_norm, W.lm_head, [L]))
    got = dec.prefill([7], KVCache(1))
    xf = x1 / math.sqrt(np.mean(x1 * x1) + TINY.rms_eps)
    assert np.allclose(got, om.widen(W.lm_head) @ xf, rtol=1e-11, atol=1e-11)


def _segment_out(dec, positions, layer=0):
    """One block over a two-token segment (tokens 5 and 9: different values, so
    the attention weights matter) that sees only itself, causally."""
    x = dec.embed([5, 9])
    out, _, _ = dec._block(layer, x, positions, lambda t, k, v: (k[:t + 1], v[:t + 1]))
    return out


def test_block_rotary_positions_are_relative(tiny):
    """RoPE on both queries and keys makes attention scores depend on the
    offset between positions only: a segment shifted as a whole gives the same
    block output, and a different gap between its two tokens does not."""
    a = _segment_out(tiny, [0, 1])
    b = _segment_out(tiny, [37, 38])
    assert np.allclose(a, b, rtol=1e-10, atol=1e-12)
    c = _segment_out(tiny, [0, 5])
    assert not np.allclose(a[1], c[1], rtol=1e-6, atol=1e-9)


def test_norm_gains_select_their_branch():
    """Each RMSNorm gain scales only its own branch: a zero attention gain
    zeroes q, k and v (so the attention branch adds exactly nothing), a zero
    FFN gain zeroes the SwiGLU input (silu(0) * 0 = 0), and a zero final gain
    zeroes the logits."""
    import copy
    W = synth.model_weights(TINY)
    x = None

    def out(attn_g, ffn_g):
        w2 = copy.copy(W)
        w2.layers = [dict(L) for L in W.layers]
        w2.layers[0]["attn_norm"] = np.full_like(W.layers[0]["attn_norm"], attn_g)
        w2.layers[0]["ffn_norm"] = np.full_like(W.layers[0]["ffn_norm"], ffn_g)
        d = Decoder(w2)
        x0 = d.embed([3])
        o, _, _ = d._block(0, x0, [2], lambda t, k, v: (k[:t + 1], v[:t + 1]))
        return x0, o

    x, o = out(0.0, 0.0)
    assert np.array_equal(o, x)
    _, o = out(0.0, 1.0)
    assert not np.allclose(o, x)
    x, o = out(1.0, 0.0)
    assert not np.allclose(o, x)
    w3 = copy.copy(W)
    w3.final_norm = np.zeros_like(W.final_norm)
    assert np.array_equal(Decoder(w3).logits(np.ones(TINY.d_model)), np.zeros(TINY.vocab))
