"""Error paths of the C ABI on a live model (tiny fp32 decoder): calls out of
order, an exhausted page pool, rows beyond the model's capacity and a
non-finite logit row are reported with their status codes, and a rejected
call leaves the state usable (the next valid call succeeds and gives the
tokens it gives without the failed call before it)."""
import numpy as np
import pytest

import synth
from tests.gpu_common import seeds_tensor, torch

pytestmark = pytest.mark.gpu
W0 = synth.TINY_FP32
E_INVALID_ARG, E_OOM, E_STATE, E_NONFINITE = 1, 2, 6, 5


@pytest.fixture(scope="module")
def rgd():
    import paper_2607_20791_amd as m
    return m


def _setup(rgd, n_pages=12, max_rows=8):
    from paper_2607_20791_amd import session
    t = torch()
    m = session.build_model(synth.model_weights(W0), max_rows=max_rows, max_pos=128)
    kv = session.alloc_kv(m, W0, max_prompts=2, max_prefix=W0.prompt_len, n_pages=n_pages)
    last = t.empty(2, W0.vocab, dtype=t.float32, device="cuda")
    rgd.prefill_kv(m, kv, session.to_device(synth.prompt_tokens(W0)[:2]), 0, last)
    return m, kv, last


def _code(rgd, fn):
    with pytest.raises(rgd.RGDError) as e:
        fn()
    return e.value.code


def test_call_order_and_capacity(rgd):
    t = torch()
    from paper_2607_20791_amd import session
    m, kv, last = _setup(rgd)
    k = 8
    ptok = t.empty(2, k, dtype=t.int32, device="cuda")
    plen = t.empty(2, dtype=t.int32, device="cuda")
    ev = t.empty(2, dtype=t.int32, device="cuda")
    table = rgd.Table([0, 3], [1, 2, 3])
    out = t.empty(1, 2, 6, dtype=t.int32, device="cuda")
    seeds = seeds_tensor(np.arange(2, dtype=np.uint64))
    # prefill again from position 0 while the prompt holds its positions
    toks = session.to_device(synth.prompt_tokens(W0)[:2])
    assert _code(rgd, lambda: rgd.prefill_kv(m, kv, toks, 0, last)) == E_STATE
    # a second probe before the gate released the first one's tails
    rgd.probe(m, kv, last, table, 2, k, 3, -1, ptok, plen, ev)
    assert _code(rgd, lambda: rgd.probe(m, kv, last, table, 2, k, 3, -1, ptok, plen, ev)) == E_STATE
    # sampling while probe tails are held
    assert _code(rgd, lambda: rgd.sample_continuations(m, kv, last, [0], 2, 6, 1.0, 0.1, seeds, out)) == E_STATE
    rgd.gate(kv, ev, 2)
    # more rows than the model holds, and min_p outside [0, 1]
    big = t.empty(1, 9, 6, dtype=t.int32, device="cuda")
    seeds9 = seeds_tensor(np.arange(9, dtype=np.uint64))
    assert _code(rgd, lambda: rgd.sample_continuations(m, kv, last, [0], 9, 6, 1.0, 0.1, seeds9, big)) == E_INVALID_ARG
    assert _code(rgd, lambda: rgd.sample_continuations(m, kv, last, [0], 2, 6, 1.0, 1.5, seeds, out)) == E_INVALID_ARG
    # the rejected calls changed nothing: sampling gives what a fresh model gives
    rgd.sample_continuations(m, kv, last, [0], 2, 6, 1.0, 0.1, seeds, out)
    m2, kv2, last2 = _setup(rgd)
    out2 = t.empty_like(out)
    rgd.sample_continuations(m2, kv2, last2, [0], 2, 6, 1.0, 0.1, seeds, out2)
    t.cuda.synchronize()
    assert t.equal(out, out2)


def test_page_pool_exhausted(rgd):
    t = torch()
    m, kv, last = _setup(rgd, n_pages=3)   # 2 rows x 40 steps need 6 pages of 16 positions
    out = t.empty(1, 2, 40, dtype=t.int32, device="cuda")
    seeds = seeds_tensor(np.arange(2, dtype=np.uint64))
    assert _code(rgd, lambda: rgd.sample_continuations(m, kv, last, [0], 2, 40, 1.0, 0.1, seeds, out)) == E_OOM
    # the pool is intact: a request that fits (1 row x 40 steps = 3 pages) runs
    one = t.empty(1, 1, 40, dtype=t.int32, device="cuda")
    rgd.sample_continuations(m, kv, last, [0], 1, 40, 1.0, 0.1, seeds[:1], one)
    t.cuda.synchronize()
    assert int(one.min()) >= 0 and int(one.max()) < W0.vocab


def test_nonfinite_logits_are_reported(rgd):
    t = torch()
    m, kv, last = _setup(rgd)
    bad = last.clone()
    bad[0, 17] = float("inf")
    out = t.empty(1, 2, 3, dtype=t.int32, device="cuda")
    seeds = seeds_tensor(np.arange(2, dtype=np.uint64))
    rgd.sample_continuations(m, kv, bad, [0], 2, 3, 1.0, 0.1, seeds, out)
    assert _code(rgd, lambda: rgd.check_status(m)) == E_NONFINITE
    rgd.check_status(m)      # the flag was cleared by the report
    rgd.sample_continuations(m, kv, last, [0], 2, 3, 1.0, 0.1, seeds, out)
    rgd.check_status(m)
