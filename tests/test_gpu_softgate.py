"""Soft compatibility gate (Appendix C) and the fixed-length probe on the GPU
vs the oracle: one probe step on identical fp32 logits at the 128256-token
vocabulary (top-K across chunks, softmax mass against rho, substitution, hard
steps after c), the tiny fp32 decoder's soft probe end to end, the probe
without a table, and the soft gate with rho > 1 reproducing the hard gate."""
import numpy as np
import pytest

import synth
from oracle import gate as ogate
from oracle import rgd as orgd
from oracle import sampler
from oracle.model import Decoder, KVCache
from tests.gpu_common import torch

pytestmark = pytest.mark.gpu
MARGIN = 1e-4
W0 = synth.TINY_FP32


@pytest.fixture(scope="module")
def rgd():
    import paper_2607_20791_amd as m
    return m


@pytest.fixture(scope="module")
def vocab_model(rgd):
    """A model with the 128256-token vocabulary of the 8B-shaped workloads
    (tiny otherwise: the probe-step hook uses only its vocabulary and
    workspace)."""
    from paper_2607_20791_amd import session
    w = synth.scaled(synth.LAYER_P8192, name="soft-mini", d_model=128, ffn=128, n_heads=1, n_kv_heads=1)
    return session.build_model(synth.model_weights(w), max_rows=64, max_pos=64)


def _csr(tables):
    offs, toks, own = [0], [], []
    for b, ents in enumerate(tables):
        for e in ents:
            toks.extend(int(x) for x in e)
            offs.append(len(toks))
            own.append(b)
    return offs, toks, own


def _fragile(info):
    """A soft step whose mass test is within the margin of rho (only when some
    alternative is compatible: an empty set fails whatever rho is)."""
    return info is not None and info.mass > 0 and info.rho_margin < MARGIN


def _planted_logits(R, V, g):
    """fp32 logits: N(0, 0.5) background plus 16 planted tokens per row whose
    probabilities (about 0.4 down to 0.004, scaled per row) make the mass of
    the top-K alternatives fall on both sides of the rho values tested."""
    w0 = np.array([8, 3, 2, 1.5, 1, 1, .8, .6, .5, .4, .3, .3, .2, .2, .1, .1])
    z = (g.normal(size=(R, V)) * 0.5).astype(np.float64)
    for r in range(R):
        ids = g.choice(V, size=16, replace=False)
        rest = np.log(np.exp(np.delete(z[r], ids)).sum())
        w = w0 * np.exp(g.normal() * 0.7)
        w[0] = w0[0]
        z[r, ids] = np.log(w) + rest
    return z.astype(np.float32)


def _step_tables(z, K, g):
    """Per row: a probe prefix q and a table that puts the step in one of the
    rule's branches (greedy compatible; alternatives in or out of the top K;
    none at all)."""
    R, V = z.shape
    states, tables = [], []
    for r in range(R):
        order = np.lexsort((np.arange(V), -z[r].astype(np.float64)))
        j = r % 3
        q = [int(x) for x in g.integers(0, V, size=j)]
        kind = r % 6
        decoy = [q + [int(g.integers(0, V))] + [1, 2]]
        if kind == 0:                               # greedy stays compatible
            ents = [q + [int(order[0]), 5, 6]]
        elif kind in (1, 2):                        # alternatives inside the top K
            picks = sorted(set(int(x) for x in g.integers(1, max(K, 2), size=2)))
            ents = [q + [int(order[p]), 7] for p in picks if p < K]
        elif kind == 3:                             # the best alternative just outside the top K
            ents = [q + [int(order[K]), 7]]
        elif kind == 4:                             # alternatives at every rank of the top K
            ents = [q + [int(order[p]), 9] for p in range(1, K)]
        else:                                       # nothing compatible
            ents = []
        states.append(q)
        tables.append(ents + decoy)
    return states, tables


@pytest.mark.parametrize("K", [1, 4, 10, 32])
@pytest.mark.parametrize("rho", [0.0, 0.02, 0.2, 1.5])
def test_probe_step_on_identical_logits(rgd, vocab_model, K, rho):
    t = torch()
    V, R, k, c = 128256, 36, 8, 2
    g = np.random.default_rng(K * 100 + int(rho * 100))
    z = _planted_logits(R, V, g)
    states, tables = _step_tables(z, K, g)
    offs, toks, own = _csr(tables)
    table = rgd.Table(offs, toks, own, min_match=2)
    ptok = np.zeros((R, k), np.int32)
    for r, q in enumerate(states):
        ptok[r, :len(q)] = q
    d_ptok = t.from_numpy(ptok).cuda()
    d_len = t.tensor([len(q) for q in states], dtype=t.int32, device="cuda")
    d_ev = t.full((R,), -1, dtype=t.int32, device="cuda")
    rgd.kernel_probe_step(vocab_model, t.from_numpy(z).cuda(), table, k, c, -1, K, rho, d_ptok, d_len, d_ev)
    t.cuda.synchronize()
    got_tok, got_len, got_ev = d_ptok.cpu().numpy(), d_len.cpu().numpy(), d_ev.cpu().numpy()
    outcomes = {"greedy": 0, "substituted": 0, "incompat": 0, "margin": 0}
    for r, q in enumerate(states):
        tok, passed, info = ogate.soft_step(q, z[r].astype(np.float64), tables[r], c, K, rho)
        if _fragile(info):
            outcomes["margin"] += 1
            continue
        j = len(q)
        ev = -1 if passed and j + 1 < k else (ogate.MAXLEN if passed else ogate.INCOMPAT)
        assert (got_tok[r, j], got_len[r], got_ev[r]) == (tok, j + 1, ev), (r, q, info)
        assert list(got_tok[r, :j]) == q
        outcomes["incompat" if not passed else ("substituted" if info is not None else "greedy")] += 1
    print(f"K={K} rho={rho}:", outcomes)
    assert outcomes["greedy"] >= R // 6
    assert outcomes["incompat"] >= R // 6
    if K > 1 and rho <= 0.02:
        assert outcomes["substituted"] >= 1


@pytest.fixture(scope="module")
def tiny():
    """The tiny fp32 decoder, its prompts' prefills and greedy sequences, and
    per-prompt tables that make the soft gate substitute: even prompts have
    an entry [y1, a] + the greedy continuation after [y1, a] (a = the second
    most probable token after the greedy first token y1), odd prompts an entry
    [y1, a5, ...] with a5 the fifth most probable."""
    weights = synth.model_weights(W0)
    dec = Decoder(weights)
    prompts = synth.prompt_tokens(W0)
    caches, last, greedy, tables = [], [], [], []
    for b in range(W0.n_prompts):
        cch = KVCache(W0.n_layers)
        lg = dec.prefill(prompts[b], cch)
        caches.append(cch)
        last.append(lg)
        y1 = sampler.argmax(lg)
        tail = KVCache(W0.n_layers)
        after = dec.decode(y1, cch, tail)
        order = np.lexsort((np.arange(len(after)), -after))
        if b % 2 == 0:
            a = int(order[1])
            seq = [y1, a]
            lg2 = dec.decode(a, cch, tail)
            while len(seq) < 6:
                seq.append(sampler.argmax(lg2))
                lg2 = dec.decode(seq[-1], cch, tail)
            tables.append([seq])
        else:
            tables.append([[y1, int(order[4]), 3, 4]])
        tail = KVCache(W0.n_layers)
        lg = last[b]
        seq = []
        while len(seq) < W0.probe_k:
            seq.append(sampler.argmax(lg))
            lg = dec.decode(seq[-1], cch, tail)
        greedy.append(seq)
    return dict(weights=weights, dec=dec, prompts=prompts, caches=caches, last=last, greedy=greedy,
                tables=tables)


def _path_margin(tiny, b, q, K):
    """Smallest argmax margin and top-K boundary gap over the logits the oracle
    probe saw for probe q of prompt b (fp32 logits of the GPU may order tokens
    differently only inside these margins)."""
    dec, cch = tiny["dec"], tiny["caches"][b]
    tail = KVCache(W0.n_layers)
    lg, worst = tiny["last"][b], np.inf
    for i in range(len(q)):
        zs = np.sort(lg)[::-1]
        worst = min(worst, zs[0] - zs[1], zs[K - 1] - zs[K])
        if i + 1 < len(q):
            lg = dec.decode(q[i], cch, tail)
    return worst


def _tiny_gpu(rgd, tiny):
    from paper_2607_20791_amd import session
    t = torch()
    m = session.build_model(tiny["weights"], max_rows=64, max_pos=128)
    kv = session.alloc_kv(m, W0, max_prompts=W0.n_prompts, max_prefix=W0.prompt_len, n_pages=96)
    B = W0.n_prompts
    last = t.empty(B, W0.vocab, dtype=t.float32, device="cuda")
    rgd.prefill_kv(m, kv, session.to_device(tiny["prompts"]), 0, last)
    return m, kv, last


def _run_probe(rgd, m, kv, last, table, soft=None):
    t = torch()
    B, k = W0.n_prompts, W0.probe_k
    ptok = t.full((B, k), -1, dtype=t.int32, device="cuda")
    plen = t.empty(B, dtype=t.int32, device="cuda")
    ev = t.empty(B, dtype=t.int32, device="cuda")
    if soft is None:
        rgd.probe(m, kv, last, table, B, k, 3, -1, ptok, plen, ev)
    else:
        rgd.probe_soft(m, kv, last, table, B, k, 3, -1, soft[0], soft[1], ptok, plen, ev)
    rgd.gate(kv, ev, B)
    return ptok.cpu().numpy(), plen.cpu().numpy(), ev.cpu().numpy()


def test_soft_probe_end_to_end_tiny(rgd, tiny):
    m, kv, last = _tiny_gpu(rgd, tiny)
    offs, toks, own = _csr(tiny["tables"])
    table = rgd.Table(offs, toks, own, min_match=2)
    K, rho, c = 4, 1e-4, 3   # the tiny model's next-token distribution is nearly flat (p ~ 1e-4)
    ptok, plen, ev = _run_probe(rgd, m, kv, last, table, (K, rho))
    hits = subs = compared = 0
    for b in range(W0.n_prompts):
        steps = []
        prefix = tiny["caches"][b]
        q, e = orgd.soft_greedy_probe(tiny["dec"], prefix, tiny["last"][b], tiny["tables"][b], W0.probe_k, c,
                                      K, rho, steps=steps)
        if any(_fragile(s) for s in steps) or _path_margin(tiny, b, q, K) < MARGIN:
            continue
        compared += 1
        assert plen[b] == len(q) and list(ptok[b, :len(q)]) == q and ev[b] == e, (b, q, e, steps)
        hits += int(ogate.is_hit(e))
        subs += sum(s.appended != s.greedy for s in steps)
    print("soft probe: compared", compared, "hits", hits, "substitutions", subs)
    assert compared >= W0.n_prompts // 2 and subs >= 1 and hits >= 1


def test_soft_gate_with_rho_above_one_is_the_hard_gate(rgd, tiny):
    m, kv, last = _tiny_gpu(rgd, tiny)
    offs, toks, own = _csr(tiny["tables"])
    table = rgd.Table(offs, toks, own, min_match=2)
    hard = _run_probe(rgd, m, kv, last, table)
    soft = _run_probe(rgd, m, kv, last, table, (8, 1.5))
    for a, b in zip(hard, soft):
        assert np.array_equal(a, b)


def test_fixed_length_probe_without_table(rgd, tiny):
    m, kv, last = _tiny_gpu(rgd, tiny)
    ptok, plen, ev = _run_probe(rgd, m, kv, last, None)
    k = W0.probe_k
    assert (plen == k).all() and (ev == ogate.MAXLEN).all()
    clean = [b for b in range(W0.n_prompts) if _path_margin(tiny, b, tiny["greedy"][b], 1) >= MARGIN]
    for b in clean:
        assert list(ptok[b]) == tiny["greedy"][b], b
    print("fixed-length probes compared:", len(clean), "of", W0.n_prompts)
    assert len(clean) >= W0.n_prompts // 2
