"""Oracle parity of the bf16 decode path at the row counts the workloads run,
and batch invariance.

The projections, the attention row blocks and the LM head pick their tile
shapes from the number of rows in a step: up to 16, 32 or 64 rows run one
row block of that height (the 8192-position layer decodes 64 branches), above
64 rows the 128-row blocks of the 8-layer workload's 128- and 256-row steps
and 256-row prefill segments.  Each shape is compared with the oracle here:
teacher-forced decode steps (logits within the bf16 tolerance on sampled rows,
every draw judged against the oracle sampler on the GPU's own logits) and a
two-prompt prefill of 300 tokens (two 256-row segments per prompt: the
last-position logits and sampled prefix K/V against the oracle's cache).

Batch invariance (Algorithm 1 samples every branch with the same S_{T,theta},
whatever else shares the step): a row's logits and tokens are bit-identical
when it runs alone and inside a 64- or 256-row step."""
import numpy as np
import pytest

import synth
from oracle import philox
from oracle import rgd as orgd
from oracle.model import Decoder, KVCache
from tests.gpu_common import Tally, judge_draw, rel_err, seeds_tensor, torch
from tests.test_gpu_path_bf16 import World

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module")
def rgd():
    import paper_2607_20791_amd as m
    return m


@pytest.fixture(scope="module")
def p512_wide(rgd):
    """The 512-position layer with room for 256-row steps."""
    return World(rgd, synth.LAYER_P512, max_rows=256)


@pytest.fixture(scope="module")
def p8192(rgd):
    return World(rgd, synth.LAYER_P8192, max_rows=64)


def run_forced(rgd, wd, forced, seeds, T, p_min):
    """Teacher-forced sampling of len(forced) rows from the prompt: returns the
    tapped logits [steps][rows][V] and the drawn tokens [rows][steps]."""
    t = torch()
    from paper_2607_20791_amd import session
    rows, steps = forced.shape
    wd.prefill(rgd)
    out = t.full((1, rows, steps), -1, dtype=t.int32, device="cuda")
    tap = t.empty(steps, rows, wd.w.vocab, dtype=t.float32, device="cuda")
    rgd.sample_continuations(wd.model, wd.kv, wd.last, [0], rows, steps, T, p_min,
                             seeds_tensor(seeds), out, forced=session.to_device(np.ascontiguousarray(forced)),
                             logits_tap=tap)
    t.cuda.synchronize()
    rgd.check_status(wd.model)
    return tap.cpu().numpy(), out.cpu().numpy()[0]


def oracle_rows(name, wd, tap, got, forced, seeds, T, p_min, check):
    """Rows `check` against the oracle: logits within TOL, draws judged."""
    tally = Tally(name)
    worst = 0.0
    steps = forced.shape[1]
    for r in check:
        br = orgd.sample_branch(wd.dec, wd.cache, wd.ref_last, int(seeds[r]), steps, T, p_min,
                                forced=forced[r], keep_logits=True)
        err = rel_err(tap[:, r], np.stack(br.logits))
        worst = max(worst, float(err.max()))
        assert err.max() <= TOL, (r, err)
        for s in range(steps):
            u = float(philox.uniform(int(seeds[r]), s))
            tally.add(judge_draw(tap[s, r], T, p_min, u, int(got[r, s])))
    return worst, tally.close()


def test_64_row_steps_8192_prefix(rgd, p8192):
    """The benchmarked step: 64 branches over the 8192-position prefix (the
    64-row GEMM tiles, split-K QKV/O/down, fused SwiGLU, two attention row
    blocks of 128 query vectors)."""
    w = p8192.w
    rows, steps = 64, 2
    forced = synth.forced_history(w, rows, steps, name="forced64")
    seeds = synth.branch_seeds(1, rows, base=900)
    tap, got = run_forced(rgd, p8192, forced, seeds, w.temperature, w.min_p)
    worst, counts = oracle_rows("8b-layer-p8192, 64-row steps, rows 0/31/63 x 2 tokens", p8192, tap, got, forced,
                                seeds, w.temperature, w.min_p, (0, 31, 63))
    print(f"8192-prefix layer, 64-row steps: logits rel err (worst) {worst:.3e}")


@pytest.mark.parametrize("rows,check", [(128, (0, 77, 127)), (256, (0, 129, 255)), (100, (0, 57, 99)),
                                       (200, (0, 131, 199))])
def test_wide_steps_512_prefix(rgd, p512_wide, rows, check):
    """128- and 256-row steps (the 8-layer workload's gated and ungated
    batches): 128-row GEMM blocks, two per weight panel at 256 rows, and four
    or eight attention row blocks (more than the four passed by value); 100
    and 200 rows: a partial 128-row block under each workgroup shape (one
    panel per wave up to 128 rows, two above)."""
    w = p512_wide.w
    steps = 2
    forced = synth.forced_history(w, rows, steps, name=f"forced{rows}")
    seeds = synth.branch_seeds(1, rows, base=1300)
    tap, got = run_forced(rgd, p512_wide, forced, seeds, w.temperature, w.min_p)
    worst, counts = oracle_rows(f"8b-layer-p512, {rows}-row steps, 3 rows x 2 tokens", p512_wide, tap, got, forced,
                                seeds, w.temperature, w.min_p, check)
    print(f"512-prefix layer, {rows}-row steps: logits rel err (worst) {worst:.3e}")


def test_multi_segment_prefill_bf16(rgd, p512_wide):
    """Two prompts of 300 tokens on a model holding 256 rows per step: each
    prompt is prefilled in a 256-row and a 44-row causal segment.  The
    last-position logits and the K/V of sampled positions (both segments,
    either side of the boundary) match the oracle's causal forward."""
    t = torch()
    from paper_2607_20791_amd import session
    wd = p512_wide
    w = synth.scaled(wd.w, name="prefill-300", n_prompts=2, prompt_len=300, synthetic_prefix=0)
    toks = synth.prompt_tokens(w)
    kv = session.alloc_kv(wd.model, w, max_prompts=2, max_prefix=300, n_pages=8)
    last = t.empty(2, w.vocab, dtype=t.float32, device="cuda")
    rgd.prefill_kv(wd.model, kv, session.to_device(toks), 0, last)
    t.cuda.synchronize()
    got_last = last.cpu().numpy()
    pk = kv.prefix_k[0].float().cpu().numpy()       # [B][Hkv][P][D]
    pv = kv.prefix_v[0].float().cpu().numpy()       # [B][Hkv][VP/64][D][64]
    worst = {"logits": 0.0, "k": 0.0, "v": 0.0}
    for b in range(2):
        cache = KVCache(1)
        ref = wd.dec.prefill(toks[b], cache)
        e = float(rel_err(got_last[b], ref))
        worst["logits"] = max(worst["logits"], e)
        assert e <= TOL, (b, e)
        Kc, Vc = cache.arrays(0)
        Kc = Kc.reshape(300, w.n_kv_heads, w.head_dim)
        Vc = Vc.reshape(300, w.n_kv_heads, w.head_dim)
        for pos in (0, 1, 150, 255, 256, 257, 299):
            gk = pk[b, :, pos, :]
            gv = pv[b, :, pos // 64, :, pos % 64]
            ek, ev = rel_err(gk, Kc[pos]).max(), rel_err(gv, Vc[pos]).max()
            worst["k"], worst["v"] = max(worst["k"], float(ek)), max(worst["v"], float(ev))
            assert ek <= TOL and ev <= TOL, (b, pos, ek, ev)
    print("300-token prefill in 256-row segments: worst rel err", worst)


def _alone_vs_batch(rgd, wd, rows, picks, name):
    w = wd.w
    steps = 3
    forced = synth.forced_history(w, rows, steps, name=name)
    seeds = synth.branch_seeds(1, rows, base=4000)
    tap, got = run_forced(rgd, wd, forced, seeds, w.temperature, w.min_p)
    for r in picks:
        tap1, got1 = run_forced(rgd, wd, forced[r:r + 1], seeds[r:r + 1], w.temperature, w.min_p)
        assert np.array_equal(tap1[:, 0], tap[:, r]), (rows, r)
        assert np.array_equal(got1[0], got[r]), (rows, r)


def test_batch_invariance_64_rows(rgd, p8192):
    """A branch alone (one-row step: 16-row tiles, 4 query vectors) against the
    same branch inside the 64-row step of the 8192-position layer."""
    _alone_vs_batch(rgd, p8192, 64, (0, 37, 63), "inv64")


def test_batch_invariance_256_rows(rgd, p512_wide):
    """A branch alone against the same branch inside a 256-row step (two
    128-row GEMM blocks, two attention row blocks) and a 64-row step."""
    _alone_vs_batch(rgd, p512_wide, 256, (5, 200), "inv256")
    _alone_vs_batch(rgd, p512_wide, 64, (5,), "inv256")
