"""The 8-layer 8B-shaped workload with 32 prompts of 1024 tokens at full size:
prefill of every prompt, a greedy probe of k=16 tokens against a shared
64-entry table in which 16 entries are the first 4 greedy tokens of the even
prompts, the gate, and 8 branches x 256 steps for every miss.

Oracle parity of this configuration is covered layer by layer by the bf16
path tests (one 8B-shaped layer at 512 and 8192 prefix positions) and end to
end by the fp32 tiny model; an fp64 oracle of 8 layers over 32 x 1024 prompt
tokens does not fit a test's time.  Here the properties of Algorithm 1 are
checked at full size: hits return the greedy sequence, the seeded prompts hit
and the others miss, a gated miss samples exactly what ungated sampling does
with the same seeds, runs are deterministic and the prompt KV is untouched.
Gated and ungated wall times are printed."""
import time

import numpy as np
import pytest

import synth
from oracle import gate as ogate
from tests.gpu_common import seeds_tensor, torch

pytestmark = pytest.mark.gpu
W4 = synth.MODEL_8LAYER


@pytest.fixture(scope="module")
def rgd():
    import paper_2607_20791_amd as m
    return m


@pytest.fixture(scope="module")
def m8(rgd):
    t = torch()
    from paper_2607_20791_amd import session
    w = W4
    B, n, k, N, S = w.n_prompts, w.prompt_len, w.probe_k, w.n_branches, w.steps
    weights = synth.model_weights(w)
    m = session.build_model(weights, max_rows=B * N, max_pos=n + S)
    pages = B * N * ((S - 1 + 15) // 16) + B * ((k - 1 + 15) // 16) + 8
    kv = session.alloc_kv(m, w, max_prompts=B, max_prefix=n, n_pages=pages)
    toks = session.to_device(synth.prompt_tokens(w))
    last = t.empty(B, w.vocab, dtype=t.float32, device="cuda")
    t.cuda.synchronize()
    t0 = time.perf_counter()
    rgd.prefill_kv(m, kv, toks, 0, last)
    t.cuda.synchronize()
    print(f"8-layer model: prefill of {B} x {n} tokens: {time.perf_counter() - t0:.3f} s")
    return dict(w=w, model=m, kv=kv, last=last, B=B, k=k, N=N, S=S)


def _ungated(rgd, c, prompts, seeds):
    t = torch()
    out = t.full((len(prompts), c["N"], c["S"]), -1, dtype=t.int32, device="cuda")
    rgd.sample_continuations(c["model"], c["kv"], c["last"], list(prompts), c["N"], c["S"], c["w"].temperature,
                             c["w"].min_p, seeds, out)
    return out


def test_8layer_gated_vs_ungated(rgd, m8):
    t = torch()
    w, m, kv, last = m8["w"], m8["model"], m8["kv"], m8["last"]
    B, k, N, S = m8["B"], m8["k"], m8["N"], m8["S"]
    before = (kv.prefix_k.clone(), kv.prefix_v.clone())
    # greedy sequences of every prompt (T = 0), used to seed the table
    greedy = t.full((B, 1, k), -1, dtype=t.int32, device="cuda")
    rgd.sample_continuations(m, kv, last, list(range(B)), 1, k, 0.0, 0.0,
                             seeds_tensor(np.arange(B, dtype=np.uint64)), greedy)
    g = greedy[:, 0].cpu().numpy()
    off, toks = synth.random_table(w, n_entries=w.n_entries - B // 2)
    ents = [list(toks[off[i]:off[i + 1]]) for i in range(len(off) - 1)]
    seeded = list(range(0, B, 2))
    ents += [list(g[b, :4]) for b in seeded]
    offs = np.concatenate([[0], np.cumsum([len(e) for e in ents])]).astype(np.int32)
    table = rgd.Table(offs, np.concatenate(ents).astype(np.int32))

    seeds_all = synth.branch_seeds(B, N)
    # gated: probe, gate, sample the misses
    t.cuda.synchronize()
    t0 = time.perf_counter()
    ptok = t.empty(B, k, dtype=t.int32, device="cuda")
    plen = t.empty(B, dtype=t.int32, device="cuda")
    ev = t.empty(B, dtype=t.int32, device="cuda")
    rgd.probe(m, kv, last, table, B, k, 3, -1, ptok, plen, ev)
    dec, miss = rgd.gate(kv, ev, B)
    miss_seeds = np.concatenate([seeds_all[b * N:(b + 1) * N] for b in miss])
    gated = _ungated(rgd, m8, miss, seeds_tensor(miss_seeds))
    t.cuda.synchronize()
    t_gated = time.perf_counter() - t0
    # ungated: every prompt sampled, no probe
    t0 = time.perf_counter()
    full = _ungated(rgd, m8, range(B), seeds_tensor(seeds_all))
    t.cuda.synchronize()
    t_ungated = time.perf_counter() - t0
    rgd.check_status(m)

    hits = [b for b in range(B) if dec[b] == 1]
    print(f"8-layer model: {len(hits)} hits, {len(miss)} misses; gated {t_gated:.3f} s "
          f"({len(miss) * N * S + sum(int(x) for x in plen.cpu()[hits])} tokens returned), "
          f"ungated {t_ungated:.3f} s ({B * N * S} tokens)")
    # the decision of each prompt follows from its greedy sequence (exact integer logic)
    ptok_h, plen_h = ptok.cpu().numpy(), plen.cpu().numpy()
    for b in range(B):
        q, e = [], ogate.MAXLEN
        for y in g[b]:
            q.append(int(y))
            if not ogate.compatible(q, ents):
                e = ogate.INCOMPAT
                break
        assert dec[b] == int(ogate.is_hit(e)), b
        assert plen_h[b] == len(q) and np.array_equal(ptok_h[b, :len(q)], g[b, :len(q)]), b
    assert set(seeded) <= set(hits) and sorted(list(miss) + hits) == list(range(B))
    full_h, gated_h = full.cpu().numpy(), gated.cpu().numpy()
    for i, b in enumerate(miss):       # a gated miss samples what ungated sampling does
        assert np.array_equal(gated_h[i], full_h[b]), b
    again = _ungated(rgd, m8, range(B), seeds_tensor(seeds_all))
    t.cuda.synchronize()
    assert t.equal(again, full)
    assert t.equal(before[0], kv.prefix_k) and t.equal(before[1], kv.prefix_v)
    assert int(full.min()) >= 0 and int(full.max()) < w.vocab
