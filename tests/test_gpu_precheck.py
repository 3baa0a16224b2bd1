"""Residual-stream classifier pre-check and the adaptive gate (Appendix A) on
the tiny fp32 decoder vs the oracle: scores at every layer within the fp32
tolerance, the prefill's logits unchanged, prompts scored <= theta skipped
(no check token, a miss) and every other prompt probed exactly as without the
pre-check (hard and soft gate)."""
import numpy as np
import pytest

import synth
from oracle import gate as ogate
from oracle import precheck
from oracle.model import Decoder, KVCache
from tests.gpu_common import torch

pytestmark = pytest.mark.gpu
W0 = synth.TINY_FP32
TOL = 1e-5


@pytest.fixture(scope="module")
def rgd():
    import paper_2607_20791_amd as m
    return m


@pytest.fixture(scope="module")
def world(rgd):
    from paper_2607_20791_amd import session
    t = torch()
    weights = synth.model_weights(W0)
    dec = Decoder(weights)
    prompts = synth.prompt_tokens(W0)
    taps = []
    for b in range(W0.n_prompts):
        tp = {}
        dec.prefill(prompts[b], KVCache(W0.n_layers), taps=tp)
        taps.append(tp)
    m = session.build_model(weights, max_rows=64, max_pos=128)
    kv = session.alloc_kv(m, W0, max_prompts=W0.n_prompts, max_prefix=W0.prompt_len, n_pages=96)
    tables, owners = [], []
    offs, toks, own = [0], [], []
    for b in range(W0.n_prompts):
        off, tok = synth.random_table(W0, f"table{b}")
        for e in ogate.table_entries(off, tok):
            toks.extend(int(x) for x in e)
            offs.append(len(toks))
            own.append(b)
    table = rgd.Table(offs, toks, own, min_match=2)
    return dict(dec=dec, prompts=prompts, taps=taps, m=m, kv=kv, table=table,
                tok=session.to_device(prompts), t=t)


def _prefill(rgd, wd, layer=None, w=None, b=0.0):
    t = wd["t"]
    B = W0.n_prompts
    last = t.empty(B, W0.vocab, dtype=t.float32, device="cuda")
    for i in range(B):
        wd["kv"].set_prefix_len(i, 0)
    if layer is None:
        rgd.prefill_kv(wd["m"], wd["kv"], wd["tok"], 0, last)
        return last, None
    scores = t.empty(B, dtype=t.float32, device="cuda")
    rgd.prefill_kv_scored(wd["m"], wd["kv"], wd["tok"], 0, last, layer, t.from_numpy(w).cuda(), b, scores)
    return last, scores


@pytest.mark.parametrize("layer", [0, 1, 2])
def test_scores_match_the_oracle(rgd, world, layer):
    t = world["t"]
    d = W0.d_model
    w = (np.random.default_rng(layer).normal(size=d) * 3 / np.sqrt(d)).astype(np.float32)
    plain, _ = _prefill(rgd, world)
    last, scores = _prefill(rgd, world, layer, w, -0.2)
    t.cuda.synchronize()
    assert t.equal(plain, last)
    got = scores.cpu().numpy()
    ref = np.array([precheck.residual_score(world["taps"][b][layer], w.astype(np.float64), -0.2)
                    for b in range(W0.n_prompts)])
    print("layer", layer, "max |score - oracle|", np.abs(got - ref).max(), "scores", np.round(got, 3))
    assert np.abs(got - ref).max() <= TOL


@pytest.mark.parametrize("topk,rho", [(0, 0.0), (4, 1e-4)])
def test_adaptive_gate_skips_low_scores(rgd, world, topk, rho):
    t = world["t"]
    B, k, d = W0.n_prompts, W0.probe_k, W0.d_model
    w = (np.random.default_rng(7).normal(size=d) * 3 / np.sqrt(d)).astype(np.float32)
    last, scores = _prefill(rgd, world, 2, w, 0.0)
    sc = scores.cpu().numpy()
    srt = np.sort(sc)
    theta = float(0.5 * (srt[B // 2 - 1] + srt[B // 2]))    # half the prompts below, none near theta
    ref = np.array([precheck.residual_score(world["taps"][b][2], w.astype(np.float64), 0.0) for b in range(B)])
    assert np.array_equal(ref <= theta, sc <= theta)
    # without the pre-check
    ptok0 = t.empty(B, k, dtype=t.int32, device="cuda")
    plen0 = t.empty(B, dtype=t.int32, device="cuda")
    ev0 = t.empty(B, dtype=t.int32, device="cuda")
    if topk:
        rgd.probe_soft(world["m"], world["kv"], last, world["table"], B, k, 3, -1, topk, rho, ptok0, plen0, ev0)
    else:
        rgd.probe(world["m"], world["kv"], last, world["table"], B, k, 3, -1, ptok0, plen0, ev0)
    rgd.gate(world["kv"], ev0, B)
    # with it
    ptok = t.empty(B, k, dtype=t.int32, device="cuda")
    plen = t.empty(B, dtype=t.int32, device="cuda")
    ev = t.empty(B, dtype=t.int32, device="cuda")
    rgd.probe_adaptive(world["m"], world["kv"], last, world["table"], B, k, 3, -1, topk, rho, scores, theta,
                       ptok, plen, ev)
    dec, miss = rgd.gate(world["kv"], ev, B)
    e0, l0, p0 = ev0.cpu().numpy(), plen0.cpu().numpy(), ptok0.cpu().numpy()
    e1, l1, p1 = ev.cpu().numpy(), plen.cpu().numpy(), ptok.cpu().numpy()
    skipped = sc <= theta
    for b in range(B):
        if skipped[b]:
            assert e1[b] == rgd.EVENT_SKIPPED and l1[b] == 0 and dec[b] == 0 and b in miss, b
        else:
            assert e1[b] == e0[b] and l1[b] == l0[b] and np.array_equal(p1[b, :l1[b]], p0[b, :l0[b]]), b
    print("skipped", int(skipped.sum()), "of", B, "misses", list(miss))
    assert 0 < skipped.sum() < B
