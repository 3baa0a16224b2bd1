"""LM-head GEMM and decode attention kernels vs the oracle on identical inputs."""
import numpy as np
import pytest

import synth
from oracle import attention as oatt
from oracle import model as om
from tests.gpu_common import bf16_to_f64, rel_err, torch

pytestmark = pytest.mark.gpu

# head layout of the Llama-3-8B layer, with a small d_model/ffn/vocab where
# the kernel under test does not depend on them
ATTN_BF16 = synth.scaled(synth.LAYER_P8192, name="attn-bf16", d_model=512, ffn=512, vocab=1024)
ATTN_F32 = synth.scaled(synth.TINY_FP32, name="attn-f32", vocab=1024)
# 8 and 16 query heads per KV head (the tail merge loops over heads per wave)
ATTN_G8 = synth.scaled(synth.LAYER_P8192, name="attn-g8", n_kv_heads=4, d_model=512, ffn=512, vocab=1024)
ATTN_G16 = synth.scaled(synth.LAYER_P8192, name="attn-g16", n_kv_heads=2, d_model=512, ffn=512, vocab=1024)


@pytest.fixture(scope="module")
def rgd():
    import paper_2607_20791_amd as m
    return m


def _model(rgd, w, max_rows, max_pos=16384):
    from paper_2607_20791_amd import session
    return session.build_model(synth.model_weights(w), max_rows=max_rows, max_pos=max_pos)


@pytest.fixture(scope="module")
def head_model(rgd):
    """A model whose LM head is the full 128256 x 4096 bf16 head of the 8B-shaped
    workloads (its other tensors are tiny and unused by this kernel)."""
    from paper_2607_20791_amd import session
    w = synth.LAYER_P8192
    head = synth.tensor(w, "lm_head", (w.vocab, w.d_model), 0.02)
    mini = synth.scaled(w, name="lm-mini", ffn=128, n_heads=1, n_kv_heads=1)
    small = synth.model_weights(synth.scaled(mini, vocab=128))
    ws = synth.Weights(mini, small.embed, small.final_norm, head, small.layers)
    return session.build_model(ws, max_rows=256, max_pos=64), head


@pytest.mark.parametrize("R", [1, 16, 37, 64, 100, 256])
def test_lm_head_bf16_full_vocab(rgd, head_model, R):
    from paper_2607_20791_amd import session
    t = torch()
    m, head = head_model
    V, d = head.shape
    g = np.random.default_rng(R)
    h = synth.to_bf16_bits(g.normal(size=(R, d)).astype(np.float32))
    logits = t.empty(R, V, dtype=t.float32, device="cuda")
    rgd.kernel_lm_head(m, session.to_device(h), logits)
    t.cuda.synchronize()
    got = logits.cpu().numpy()
    rows = sorted({0, R // 2, R - 1} | ({63, 64, 127, 128, 200} & set(range(R))))
    want = om.linear(head, om.widen(h[rows]))
    err = rel_err(got[rows], want)
    print("lm head rel err", err.max())
    assert err.max() <= 2e-2
    assert err.max() <= 1e-4   # identical bf16 inputs: only the fp32 accumulation order differs


def _attn_case(rgd, w, m, R_per_prompt, prompts, P, tail, plens=None, splits=0, seed=0):
    t = torch()
    from paper_2607_20791_amd import session
    g = np.random.default_rng(seed)
    Hq, Hkv, D = w.n_heads, w.n_kv_heads, w.head_dim
    R = R_per_prompt * prompts
    cast = synth.to_bf16_bits if w.dtype == "bf16" else (lambda a: a.astype(np.float32))
    q = cast(g.normal(size=(R, Hq, D)).astype(np.float32))
    kp = cast(g.normal(size=(prompts, P, Hkv, D)).astype(np.float32))
    vp = cast(g.normal(size=(prompts, P, Hkv, D)).astype(np.float32))
    ps = 16
    npg = (tail + ps - 1) // ps
    n_pages = R * max(npg, 1) + 3
    pool_k = cast(g.normal(size=(n_pages, ps, Hkv, D)).astype(np.float32))
    pool_v = cast(g.normal(size=(n_pages, ps, Hkv, D)).astype(np.float32))
    perm = g.permutation(n_pages)[:R * max(npg, 1)].reshape(R, max(npg, 1)).astype(np.int32)
    row_prompt = np.repeat(np.arange(prompts), R_per_prompt).astype(np.int32)
    plen = np.full(R, P, np.int32) if plens is None else np.asarray(plens, np.int32)
    out = t.empty(R, Hq * D, dtype=t.bfloat16 if w.dtype == "bf16" else t.float32, device="cuda")
    dev = session.to_device
    # cache layouts: prefix K [prompts][Hkv][P][D], V [prompts][Hkv][VP/64][D][64];
    # pages K [page][Hkv][ps][D], V [page][Hkv][D][ps]
    VP = session.v_stride(P)
    kp_c = session.k_cache_layout(kp)
    vp_c = session.v_cache_layout(vp, VP)
    pool_k_c = np.ascontiguousarray(pool_k.transpose(0, 2, 1, 3))
    pool_v_c = np.ascontiguousarray(pool_v.transpose(0, 2, 3, 1))
    rgd.kernel_attention(m, dev(q), row_prompt, plen, dev(kp_c), dev(vp_c), prompts, P, dev(pool_k_c),
                         dev(pool_v_c), ps, dev(perm), perm.shape[1], tail, out, splits=splits)
    t.cuda.synchronize()
    got = (bf16_to_f64(out) if w.dtype == "bf16" else out.cpu().numpy()).reshape(R, Hq, D)
    W = om.widen
    errs = []
    for r in range(R):
        b = row_prompt[r]
        kt = np.concatenate([W(pool_k[p]) for p in perm[r]])[:tail] if tail else np.zeros((0, Hkv, D))
        vt = np.concatenate([W(pool_v[p]) for p in perm[r]])[:tail] if tail else np.zeros((0, Hkv, D))
        ref = oatt.attend_prefix_tail(W(q[r]), W(kp[b, :plen[r]]), W(vp[b, :plen[r]]), kt, vt)
        errs.append(rel_err(got[r], ref).max())
    return np.array(errs)


@pytest.fixture(scope="module")
def mb(rgd):
    return _model(rgd, ATTN_BF16, max_rows=64)


@pytest.mark.parametrize("R,prompts,P,tail", [(1, 1, 8193, 0), (1, 1, 8193, 15), (16, 1, 513, 37),
                                              (64, 1, 8193, 37), (8, 3, 300, 16), (5, 2, 31, 1)])
def test_attention_bf16(rgd, mb, R, prompts, P, tail):
    err = _attn_case(rgd, ATTN_BF16, mb, R, prompts, P, tail, seed=R + P + tail)
    print("attention bf16 rel err", err.max())
    assert err.max() <= 2e-2


def test_attention_bf16_causal_rows_and_forced_splits(rgd, mb):
    plens = list(range(90, 130, 2))   # 20 rows of one prompt with increasing visible prefix
    err = _attn_case(rgd, ATTN_BF16, mb, 20, 1, 130, 0, plens=plens, splits=3, seed=5)
    assert err.max() <= 2e-2
    err1 = _attn_case(rgd, ATTN_BF16, mb, 4, 1, 4000, 20, splits=1, seed=6)
    err9 = _attn_case(rgd, ATTN_BF16, mb, 4, 1, 4000, 20, splits=9, seed=6)
    assert err1.max() <= 2e-2 and err9.max() <= 2e-2


def test_attention_bf16_long_tail_and_many_splits(rgd, mb):
    # tail of 300 positions: each wave of the merge kernel attends several tiles
    err = _attn_case(rgd, ATTN_BF16, mb, 4, 1, 700, 300, seed=11)
    assert err.max() <= 2e-2
    # more prefix splits than the merge kernel prefetches (16): the rest are
    # loaded by the combine of the split partials
    err = _attn_case(rgd, ATTN_BF16, mb, 4, 1, 8193, 5, splits=40, seed=12)
    assert err.max() <= 2e-2


@pytest.mark.parametrize("w", [ATTN_G8, ATTN_G16], ids=["G8", "G16"])
def test_attention_bf16_wide_groups(rgd, w):
    m = _model(rgd, w, max_rows=64)
    for R, prompts, P, tail in [(32, 1, 1000, 40), (3, 2, 200, 7)]:
        err = _attn_case(rgd, w, m, R, prompts, P, tail, seed=R + P)
        assert err.max() <= 2e-2, (R, prompts, P, tail, err.max())


def test_fill_prefix_round_trip(rgd, mb):
    from paper_2607_20791_amd import session
    t = torch()
    w = ATTN_BF16
    kv = session.alloc_kv(mb, w, max_prompts=2, max_prefix=100, n_pages=4)
    g = np.random.default_rng(3)
    k = synth.to_bf16_bits(g.normal(size=(2, 90, w.n_kv_heads, w.head_dim)).astype(np.float32))
    v = synth.to_bf16_bits(g.normal(size=(2, 90, w.n_kv_heads, w.head_dim)).astype(np.float32))
    session.fill_prefix(kv, 0, k, v)
    t.cuda.synchronize()
    pk = kv.prefix_k[0].view(t.int16).cpu().numpy().view(np.uint16)
    pv = kv.prefix_v[0].view(t.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(pk[:, :, :90], session.k_cache_layout(k))
    assert np.array_equal(pv, session.v_cache_layout(v, session.v_stride(100)))


@pytest.fixture(scope="module")
def mf(rgd):
    return _model(rgd, ATTN_F32, max_rows=64, max_pos=2048)


@pytest.mark.parametrize("R,prompts,P,tail", [(1, 1, 65, 0), (4, 2, 64, 31), (16, 1, 600, 300)])
def test_attention_f32(rgd, mf, R, prompts, P, tail):
    err = _attn_case(rgd, ATTN_F32, mf, R, prompts, P, tail, seed=P + tail)
    print("attention f32 rel err", err.max())
    assert err.max() <= 1e-5
