#!/usr/bin/env python3
"""Benchmark of the refusal-gated decode hot path on one MI355X.

Workload: one Llama-3-8B-shaped decoder layer in bf16 (d=4096, 32/8 heads,
D=128, SwiGLU 14336, vocab 128256, random init) over a shared prompt KV of 8192
synthetic N(0,1) positions plus one prefilled last prompt token; a greedy probe
of up to k=16 tokens against a 64-entry refusal table; the gate; and N=64
min-p branches (T=2.0, min_p=0.05) of 128 tokens each on paged tails.

One step = prefill of the last prompt token + probe + gate + (on a miss) all
sampling steps.  `value` counts decoded tokens (probe tokens + branch tokens)
per second over the timed steps.  Kernel durations come from HIP events the
library records on its own stream during the timed sampling calls.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "gated decode tokens/sec (probe+N branches) + % HBM roofline, attn & sampler"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
# the library times decode steps 1, 1+P, 1+2P, ... of each sampling call
# (P = TIMING_PERIOD), one unit per timed step in turn (LM head, attention
# stage, prefix attention kernel, sampler, whole step); the other steps run
# without event records
TIMING_PERIOD = 4
TIMER_UNITS = ("lm_head", "attention", "attn_prefix", "sampler", "step")


def timed_steps(n_decode, unit):
    """Indices i (decode step i + 1) of the steps of one sampling call on which
    the library timed `unit`."""
    u = TIMER_UNITS.index(unit)
    return [i for i in range(n_decode) if i % TIMING_PERIOD == 0 and (i // TIMING_PERIOD) % len(TIMER_UNITS) == u]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def measured_traffic(name="lm_head_8b_layer_p8192_traffic.md"):
    """HBM bytes per launch from the committed counter summary, or None when
    the kernel source changed since the counters were taken."""
    import hashlib
    import re
    try:
        text = open(os.path.join(ROOT, "profiles", name)).read()
        block = re.search(r"```traffic\n(.*?)```", text, re.S).group(1)
        kv = dict(line.split("=", 1) for line in block.strip().splitlines())
        src = open(os.path.join(ROOT, kv["source"]), "rb").read()
        if hashlib.sha256(src).hexdigest() != kv["sha256"]:
            return None
        return int(kv["bytes_per_launch"])
    except Exception:  # pragma: no cover
        return None


SOFT_TOPK, SOFT_RHO = 10, 0.1


def gate_variants(rgd, torch, model, kv, w, last, last_tok, table, prefill, k, c, sampling_ms, reps=5):
    """Probe + gate wall time (median of `reps`, ms) of the hard gate, the soft
    compatibility gate (top-10, rho = 0.1) and the fixed-length probe (no
    table), on the typical table and on an adversarial one (an entry equal to
    the first k-1 greedy tokens and different at token k: a full-length miss),
    each also as a fraction of ungated sampling time per step; and the cost of
    the residual-stream pre-check (its readout inside the prefill, and probe +
    gate of a prompt it skips)."""
    import statistics
    import numpy as np
    dev = "cuda"
    ptok = torch.empty(1, k, dtype=torch.int32, device=dev)
    plen = torch.empty(1, dtype=torch.int32, device=dev)
    ev = torch.empty(1, dtype=torch.int32, device=dev)
    prefill()
    torch.cuda.synchronize()

    def timed(fn):
        ts = []
        for _ in range(reps):
            t0 = time.perf_counter()
            fn()
            rgd.gate(kv, ev, 1)
            ts.append((time.perf_counter() - t0) * 1e3)
        return statistics.median(ts), int(plen.item()), int(ev.item())

    g = torch.empty(1, 1, k, dtype=torch.int32, device=dev)
    rgd.sample_continuations(model, kv, last, [0], 1, k, 0.0, 0.0, torch.zeros(1, dtype=torch.int64, device=dev), g)
    gl = g[0, 0].cpu().numpy()
    adv = rgd.Table(np.array([0, k], np.int32), np.array(list(gl[:k - 1]) + [int((gl[k - 1] + 1) % w.vocab)],
                                                        np.int32))
    out = {"soft_topk": SOFT_TOPK, "soft_rho": SOFT_RHO, "sampling_ms_per_step": round(sampling_ms, 3)}
    cases = {
        "hard_typical": lambda: rgd.probe(model, kv, last, table, 1, k, c, -1, ptok, plen, ev),
        "soft_typical": lambda: rgd.probe_soft(model, kv, last, table, 1, k, c, -1, SOFT_TOPK, SOFT_RHO,
                                               ptok, plen, ev),
        "hard_adversarial": lambda: rgd.probe(model, kv, last, adv, 1, k, c, -1, ptok, plen, ev),
        "soft_adversarial": lambda: rgd.probe_soft(model, kv, last, adv, 1, k, c, -1, SOFT_TOPK, SOFT_RHO,
                                                   ptok, plen, ev),
        "fixed_length": lambda: rgd.probe(model, kv, last, None, 1, k, c, -1, ptok, plen, ev),
    }
    for name, fn in cases.items():
        ms, n, e = timed(fn)
        out[name] = {"probe_gate_ms": round(ms, 3), "probe_tokens": n, "event": e,
                     "overhead": round(ms / sampling_ms, 5) if sampling_ms > 0 else None}

    # probes without early exit, the table applied to the finished probe
    # (rgd_probe_fixed): the fixed-probe ablation (Appendix B, 32 greedy tokens)
    # and the naive greedy-then-high-temperature approach (Section 3, up to 128
    # greedy tokens); on the typical table both are misses, so the prompt is then
    # sampled as without a gate.  Cost row in the style of Table 1: check tokens,
    # added latency and the ratio of gated to direct latency.
    for name, kk in (("fixed_probe_k32", 32), ("naive_k128", 128)):
        pt = torch.empty(1, kk, dtype=torch.int32, device=dev)
        ms, n, e = timed(lambda: rgd.probe_fixed(model, kv, last, table, 1, kk, c, -1, pt, plen, ev))
        out[name] = {"probe_gate_ms": round(ms, 3), "probe_tokens": n, "event": e,
                     "miss": e in (0, 3), "delta_ms": round(ms, 3),
                     "ratio_vs_direct": round((ms + sampling_ms) / sampling_ms, 4) if sampling_ms > 0 else None}

    # residual-stream pre-check (random classifier weights: the cost, not the accuracy): the
    # prefill with and without the readout, and probe + gate of a prompt it skips (theta = 1)
    d = w.d_model
    cls_w = torch.from_numpy((np.random.default_rng(0).normal(size=d) / np.sqrt(d)).astype(np.float32)).to(dev)
    scores = torch.empty(1, dtype=torch.float32, device=dev)
    tok = torch.tensor([[int(last_tok)]], dtype=torch.int32, device=dev)

    def pf(scored):
        kv.set_prefix_len(0, w.synthetic_prefix)
        if scored:
            rgd.prefill_kv_scored(model, kv, tok, w.synthetic_prefix, last, w.n_layers, cls_w, 0.0, scores)
        else:
            rgd.prefill_kv(model, kv, tok, w.synthetic_prefix, last)
        torch.cuda.synchronize()

    def med(fn, n=reps * 2):
        ts = []
        for _ in range(n):
            t0 = time.perf_counter()
            fn()
            ts.append((time.perf_counter() - t0) * 1e3)
        return statistics.median(ts)
    plain_ms, scored_ms = med(lambda: pf(False)), med(lambda: pf(True))
    skip_ms, n, e = timed(lambda: rgd.probe_adaptive(model, kv, last, table, 1, k, c, -1, 0, 0.0, scores, 1.0,
                                                     ptok, plen, ev))
    out["precheck"] = {"layer": w.n_layers, "prefill_ms": round(plain_ms, 3), "prefill_scored_ms": round(scored_ms, 3),
                       "skipped_probe_gate_ms": round(skip_ms, 3), "probe_tokens": n, "event": e,
                       "overhead": round(skip_ms / sampling_ms, 5) if sampling_ms > 0 else None}
    return out


def algorithmic(w, R, P, tails):
    """Algorithmic bytes / flops per launch of the three named kernels."""
    d, V, Hq, Hkv, D = w.d_model, w.vocab, w.n_heads, w.n_kv_heads, w.head_dim
    ntiles = (V + 511) // 512   # row maxima the LM head emits (one per 512-column group)
    lm_bytes = V * d * 2 + R * d * 2 + R * V * 4 + R * ntiles * 4
    lm_flops = 2.0 * R * d * V
    att_bytes = [2 * P * Hkv * D * 2 + R * 2 * t * Hkv * D * 2 + 2 * R * Hq * D * 2 for t in tails]
    att_flops = [4.0 * R * Hq * D * (P + t) for t in tails]
    samp_bytes = R * V * 4 + R * ntiles * 4
    return lm_bytes, lm_flops, att_bytes, att_flops, samp_bytes


def sampler_sweep(rgd, torch, reps=20, flush_mode="read"):
    """The standalone min-p sampler on the sampler-sweep workload (256 rows of
    152064 Zipf-biased logits) at every (T, p_min) grid point, plus T = 0
    (argmax): median time of `reps` calls, each timed alone with events on the
    launch stream after a 512 MiB write that evicts the logits from the
    last-level cache (the 155.7 MB of logits would otherwise stay resident in
    it from one call to the next).  Algorithmic bytes per call: the logits
    once plus the tokens."""
    import synth
    s = synth.SWEEP
    z = torch.from_numpy(synth.sweep_logits(s)).cuda()
    R, V = z.shape
    ws = torch.empty(rgd.sampler_workspace_bytes(R, V), dtype=torch.uint8, device="cuda")
    out = torch.empty(R, 1, dtype=torch.int32, device="cuda")
    seeds = torch.arange(R, dtype=torch.int64, device="cuda")
    nbytes = R * V * 4 + R * 4

    flush = torch.ones(128 << 20, dtype=torch.float32, device="cuda")
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]

    def evict():
        if flush_mode == "read":
            flush.max()
        elif flush_mode == "write":
            flush.fill_(1)

    def timed(f):
        for _ in range(3):
            f()
        for e0, e1 in ev:
            evict()
            e0.record()
            f()
            e1.record()
        torch.cuda.synchronize()
        t = sorted(e0.elapsed_time(e1) * 1e3 for e0, e1 in ev)
        return t[len(t) // 2]

    pts = []
    for T in s.temperatures:
        for pm in s.min_ps:
            us = timed(lambda: rgd.kernel_sample(z, T, pm, seeds, 0, 0, 1, ws, out))
            pts.append({"T": T, "min_p": pm, "us": round(us, 2)})
    am = timed(lambda: rgd.kernel_argmax(z, ws, out[:, 0]))
    pl = [{"T": T, "us": round(timed(lambda: rgd.kernel_sample_pless(z, T, seeds, 0, 0, 1, ws, out)), 2)}
          for T in s.temperatures]
    us_all = sorted(p["us"] for p in pts)
    med = us_all[len(us_all) // 2]
    pl_med = sorted(p["us"] for p in pl)[len(pl) // 2]
    return {"workload": s.name, "rows": R, "vocab": V, "bytes_per_call": nbytes, "points": pts,
            "median_us": med, "median_gbs": round(nbytes / (med * 1e-6) / 1e9, 1),
            "median_frac": round(nbytes / (med * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "argmax_us": round(am, 2),
            "pless": {"points": pl, "median_us": pl_med,
                      "median_frac": round(nbytes / (pl_med * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}}


def pless_variant(rgd, torch, model, kv, w, last, N, S, seeds, out, minp_ms, reps=3):
    """The same N x S sampling call with p-less truncation (keep p_i >= sum_j
    p_j^2 of softmax(z/T), the truncation of the paper's experiments) in place
    of min-p: wall time per call (device synchronisations around it), tokens/s,
    and the library's event timings of the p-less sampler and of a decode
    step.  Algorithmic sampler bytes: the logits once (R x V x 4); the kernels
    read them twice (statistics, then the chunks above the threshold)."""
    def run(timed):
        if timed:
            rgd.timing_enable(model, TIMING_PERIOD)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        rgd.sample_continuations_pless(model, kv, last, [0], N, S, w.temperature, seeds, out)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        if timed:
            rgd.timing_enable(model, 0)
        return dt

    run(False)
    rgd.timing_read(model)
    ts = sorted(run(True) for _ in range(reps))
    rgd.check_status(model)
    tim = rgd.timing_read(model)
    sp_ms, sp_n = tim["sampler"]
    st_ms, st_n = tim["step"]
    med = ts[len(ts) // 2]
    sb = N * w.vocab * 4
    sp_us = sp_ms / sp_n * 1e3
    return {"sampling_ms": round(med * 1e3, 3), "tokens_per_s": round(N * S / med, 1),
            "vs_minp_sampling": round(med * 1e3 / minp_ms, 4),
            "sampler_avg_us": round(sp_us, 2), "sampler_gbs": round(sb / (sp_us * 1e-6) / 1e9, 1),
            "sampler_frac": round(sb / (sp_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "decode_step_avg_us": round(st_ms / st_n * 1e3, 2)}


def cpu_baseline(weights, w, P, last_tok, kp, vp, budget_s=15.0):
    """The oracle on the host: prefill of the last prompt token, then one
    branch's draws and decode steps until the time budget is spent."""
    import numpy as np
    from oracle import philox, sampler
    from oracle.model import Decoder, KVCache
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    dec = Decoder(weights)
    cache = KVCache.from_arrays([kp[0]], [vp[0]])
    t0 = time.perf_counter()
    logits = dec.prefill([int(last_tok)], cache, start_pos=P)
    tail = KVCache(w.n_layers)
    n = 0
    while True:
        u = float(philox.uniform(12345, n))
        d = sampler.sample_minp(logits, w.temperature, w.min_p, u)
        n += 1
        if time.perf_counter() - t0 > budget_s or n >= w.steps:
            break
        logits = dec.decode(d.token, cache, tail)
    el = time.perf_counter() - t0
    return {"value": n / el, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"prefill of the last prompt token over the 8192-position prefix, then {n} "
                      f"min-p draws and {n - 1} decode steps of one branch (float64 numpy), "
                      f"{el:.1f} s"}


def eight_layer(rgd, torch, reps):
    """The 8-layer 8B-shaped model, 32 prompts of 1024 tokens (prefill timed on
    its own), a shared 64-entry table in which 16 entries are the first 4 greedy
    tokens of the even prompts, and 8 branches x 256 min-p tokens (T=2,
    p_min=0.1) per miss.  Gated (probe k=16, c=3, gate, sampling of the misses)
    against ungated (every prompt sampled, no probe) wall time, median of reps,
    with the cost row of the miss prompts: the check tokens they decoded, the
    probe + gate time, and the ratio of gated to direct latency for them."""
    import numpy as np
    import synth
    from paper_2607_20791_amd import session
    w = synth.MODEL_8LAYER
    B, n, k, N, S = w.n_prompts, w.prompt_len, w.probe_k, w.n_branches, w.steps
    log("8-layer model: weights ...")
    m = session.build_model(synth.model_weights(w), max_rows=B * N, max_pos=n + S)
    pages = B * N * ((S - 1 + 15) // 16) + B * ((k - 1 + 15) // 16) + 8
    kv = session.alloc_kv(m, w, max_prompts=B, max_prefix=n, n_pages=pages)
    toks = session.to_device(synth.prompt_tokens(w))
    last = torch.empty(B, w.vocab, dtype=torch.float32, device="cuda")
    log("8-layer model: prefill ...")
    rgd.prefill_kv(m, kv, toks, 0, last)
    torch.cuda.synchronize()
    for b in range(B):            # the timed prefill rewrites the same prompt KV
        kv.set_prefix_len(b, 0)
    t0 = time.perf_counter()
    rgd.prefill_kv(m, kv, toks, 0, last)
    torch.cuda.synchronize()
    prefill_s = time.perf_counter() - t0
    greedy = torch.full((B, 1, k), -1, dtype=torch.int32, device="cuda")
    rgd.sample_continuations(m, kv, last, list(range(B)), 1, k, 0.0, 0.0,
                             torch.arange(B, dtype=torch.int64, device="cuda"), greedy)
    g = greedy[:, 0].cpu().numpy()
    off, tk = synth.random_table(w, n_entries=w.n_entries - B // 2)
    ents = [list(tk[off[i]:off[i + 1]]) for i in range(len(off) - 1)]
    ents += [list(g[b, :4]) for b in range(0, B, 2)]
    offs = np.concatenate([[0], np.cumsum([len(e) for e in ents])]).astype(np.int32)
    table = rgd.Table(offs, np.concatenate(ents).astype(np.int32))
    seeds_all = torch.from_numpy(synth.branch_seeds(B, N).view(np.int64)).cuda()
    ptok = torch.empty(B, k, dtype=torch.int32, device="cuda")
    plen = torch.empty(B, dtype=torch.int32, device="cuda")
    ev = torch.empty(B, dtype=torch.int32, device="cuda")
    out = torch.empty(B, N, S, dtype=torch.int32, device="cuda")

    def rows_of(prompts):
        return torch.tensor([b * N + j for b in prompts for j in range(N)], dtype=torch.int64, device="cuda")

    def gated():
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        rgd.probe(m, kv, last, table, B, k, 3, -1, ptok, plen, ev)
        dec, miss = rgd.gate(kv, ev, B)
        t1 = time.perf_counter()
        if len(miss):
            rgd.sample_continuations(m, kv, last, list(miss), N, S, w.temperature, w.min_p,
                                     seeds_all[rows_of(miss)], out[:len(miss)])
        torch.cuda.synchronize()
        return time.perf_counter() - t0, t1 - t0, list(dec), list(miss)

    def ungated(prompts):
        sd = seeds_all[rows_of(prompts)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        rgd.sample_continuations(m, kv, last, list(prompts), N, S, w.temperature, w.min_p, sd, out[:len(prompts)])
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    log("8-layer model: gated and ungated runs ...")
    gated()
    runs = sorted((gated() for _ in range(reps)), key=lambda r: r[0])
    t_g, t_pg, dec, miss = runs[len(runs) // 2]
    t_u = sorted(ungated(range(B)) for _ in range(reps))[reps // 2]
    t_um = sorted(ungated(miss) for _ in range(reps))[reps // 2] if miss else 0.0
    # one more ungated call with the library timers on: the LM head and the
    # whole decode step at B x N rows
    rgd.timing_enable(m, 1)
    rgd.timing_enable(m, 0)
    rgd.timing_read(m)
    rgd.timing_enable(m, TIMING_PERIOD)
    ungated(range(B))
    rgd.timing_enable(m, 0)
    tim = rgd.timing_read(m)
    rgd.check_status(m)
    pl = plen.cpu().numpy()
    hits = [b for b in range(B) if dec[b] == 1]
    returned = len(miss) * N * S + int(sum(int(pl[b]) for b in hits))
    # Byte model of one ungated decode step (B x N rows): every layer's weights
    # and the LM head once, each prompt's KV once per layer, each row's tail
    # (on average (S + 1) / 2 positions) once per layer, the logits written and
    # read once; bf16 weights and KV, fp32 logits.
    R = B * N
    qkv = (w.n_heads + 2 * w.n_kv_heads) * w.head_dim
    layer_w = (qkv * w.d_model + w.n_heads * w.head_dim * w.d_model + 3 * w.ffn * w.d_model) * 2
    kv_pos = w.n_kv_heads * w.head_dim * 2 * 2
    step_bytes = (w.n_layers * layer_w + w.vocab * w.d_model * 2 + w.n_layers * B * n * kv_pos
                  + w.n_layers * R * (S + 1) / 2 * kv_pos + R * w.vocab * 4 * 2)
    ceiling = R / (step_bytes / (HBM_PEAK_GBS * 1e9))
    lm_bytes = w.vocab * w.d_model * 2 + R * w.d_model * 2 + R * w.vocab * 4
    lm_us = tim["lm_head"][0] / max(tim["lm_head"][1], 1) * 1e3
    step_us = tim["step"][0] / max(tim["step"][1], 1) * 1e3
    return {"workload": w.name, "prompts": B, "prompt_len": n, "branches": N, "steps": S, "probe_k": k,
            "hits": len(hits), "misses": len(miss), "prefill_s": round(prefill_s, 4),
            "gated_s": round(t_g, 4), "gated_tokens_returned": returned,
            "gated_tokens_per_s": round(returned / t_g, 1),
            "ungated_s": round(t_u, 4), "ungated_tokens": B * N * S,
            "ungated_tokens_per_s": round(B * N * S / t_u, 1),
            "miss_cost": {"check_tokens_per_miss": round(float(np.mean([pl[b] for b in miss])), 3) if miss else None,
                          "probe_gate_ms": round(t_pg * 1e3, 3),
                          "direct_sampling_of_misses_ms": round(t_um * 1e3, 3),
                          "ratio": round((t_pg + t_um) / t_um, 4) if t_um > 0 else None},
            "byte_model": {"ungated_bytes_per_step": int(step_bytes),
                           "ungated_ceiling_tokens_per_s": round(ceiling, 1),
                           "ungated_frac": round(B * N * S / t_u / ceiling, 4),
                           "decode_step_us": round(step_us, 2),
                           "decode_step_frac": round(step_bytes / (step_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                           "lm_head_us": round(lm_us, 2),
                           "lm_head_frac": round(lm_bytes / (lm_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}}


def cpu_baseline_units(reps=3):
    """The CPU-baseline leg per unit: the oracle (float64 numpy, this host's
    BLAS threads) timed on the units of the workloads, each on a bounded
    sample that is stated.  Sampler rows of the sampler sweep at every
    (T, p_min) point and argmax; attention and LM head of one decode step at
    the 512- and 8192-position layers (t = 1); one whole decode step of one row
    of the 512-position layer; the tiny fp32 decoder's refusal-gated run of one
    prompt; and the LM head again on one thread."""
    import platform
    import statistics
    import numpy as np
    import synth
    from oracle import attention, philox, sampler
    from oracle import rgd as orgd
    from oracle.model import Decoder, KVCache, linear
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threadpool_limits, threads = None, os.cpu_count() or 1
    cpu = platform.processor() or "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass

    def med(fn, n=reps):
        ts = []
        for _ in range(n):
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return statistics.median(ts)

    out = {"kind": "oracle", "cpu": cpu, "logical_cpus": os.cpu_count(), "blas_threads": int(threads)}
    # sampler rows (152064 logits)
    z = synth.sweep_logits(synth.SWEEP, rows=2)
    s = synth.SWEEP
    pts = []
    for T in s.temperatures:
        for pm in s.min_ps:
            u = float(philox.uniform(0, 0))
            pts.append({"T": T, "min_p": pm, "ms_per_row": round(med(lambda: sampler.sample_minp(z[0], T, pm, u)) * 1e3, 3)})
    out["sampler_row_ms"] = pts
    out["argmax_row_ms"] = round(med(lambda: sampler.argmax(z[0])) * 1e3, 3)
    log("oracle units: 8B-shaped layer weights ...")
    w1 = synth.LAYER_P512
    weights = synth.model_weights(w1)
    dec = Decoder(weights)
    g = np.random.default_rng(0)
    for name, P, R in (("p512", 513, 16), ("p8192", 8193, 64)):
        q = g.normal(size=(32, 128))
        k = g.normal(size=(P + 1, 8, 128))
        v = g.normal(size=(P + 1, 8, 128))
        rows = 2
        t = med(lambda: [attention.attend(q, k, v) for _ in range(rows)], n=1)
        out[f"attention_step_{name}_ms"] = round(t / rows * R * 1e3, 1)
        out[f"attention_step_{name}_sample"] = f"{rows} of the {R} rows timed, scaled to {R}"
        x = g.normal(size=(R, 4096))
        out[f"lm_head_step_{name}_ms"] = round(med(lambda: linear(weights.lm_head, x), n=1) * 1e3, 1)
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            x = g.normal(size=(16, 4096))
            out["lm_head_step_p512_1thread_ms"] = round(med(lambda: linear(weights.lm_head, x), n=1) * 1e3, 1)
    # one decode step of one row of the 512-position layer (prefix of 512 N(0,1) positions)
    kp, vp = synth.synthetic_prefix_kv(w1, 0)
    cache = KVCache.from_arrays([kp[0]], [vp[0]])
    last_tok = int(synth.prompt_tokens(w1)[0, 0])
    dec.prefill([last_tok], cache, start_pos=w1.synthetic_prefix)
    tail = KVCache(1)
    out["decode_step_p512_one_row_ms"] = round(med(lambda: dec.decode(7, cache, tail), n=2) * 1e3, 1)
    # the tiny fp32 decoder: refusal-gated decoding of one prompt (prefill, probe, gate, 1 x 32 draws)
    w0 = synth.TINY_FP32
    d0 = Decoder(synth.model_weights(w0))
    p0 = synth.prompt_tokens(w0)[1]
    off, tk = synth.random_table(w0, "table1")
    ents = [list(tk[off[i]:off[i + 1]]) for i in range(len(off) - 1)]
    out["tiny_gated_one_prompt_s"] = round(med(lambda: orgd.refusal_gated(d0, p0, ents, w0.probe_k, [1], w0.steps,
                                                                       w0.temperature, w0.min_p), n=1), 2)
    # the 8-layer 32-prompt workload, extrapolated (the oracle decodes one row at a time): one
    # layer of a one-row step = the one-row decode step minus the LM head (whose cost hardly
    # depends on the rows), times 8 layers, plus the LM head; ungated = every prompt's 8 x 256
    w4 = synth.MODEL_8LAYER
    layer_s = max(out["decode_step_p512_one_row_ms"] - out["lm_head_step_p512_ms"], 0.0) / 1e3
    row_step_s = w4.n_layers * layer_s + out["lm_head_step_p512_ms"] / 1e3
    out["eight_layer_extrapolated"] = {
        "row_step_s": round(row_step_s, 3),
        "ungated_hours": round(w4.n_prompts * w4.n_branches * w4.steps * row_step_s / 3600, 1),
        "basis": "extrapolated from the measured one-row decode step and LM head of one 8B-shaped layer"}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=8)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--table", choices=("typical", "adversarial"), default="typical")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-eight-layer", action="store_true",
                    help="leave out the 8-layer gated-vs-ungated run of the default line")
    ap.add_argument("--workload", choices=("8b-layer-p8192", "8b-8layer-32x1024"), default="8b-layer-p8192",
                    help="the default (one 8B-shaped layer, 8192-position prefix, 64 x 128 branches) or the "
                         "8-layer model with 32 prompts (gated vs ungated wall time, its own JSON line)")
    ap.add_argument("--oracle-units", action="store_true",
                    help="only time the oracle per unit on the host (the CPU-baseline leg; no GPU needed)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device copy (scales the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (got --gpus {args.gpus}); the path is built and "
              "measured on one MI355X only", file=sys.stderr)
        sys.exit(2)

    if args.oracle_units:
        print(json.dumps(cpu_baseline_units()), flush=True)
        return

    import numpy as np
    import torch

    if args.calibrate_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_per_launch": 1 << 30, "launches": 3}))
        return

    if args.workload == "8b-8layer-32x1024":
        import paper_2607_20791_amd as rgd
        res = eight_layer(rgd, torch, reps=max(1, args.steps // 4))
        print(json.dumps({"metric": "gated vs ungated wall time (8-layer, 32 prompts)",
                          "value": res["gated_tokens_per_s"], "unit": "tokens/s", "n_gpus": 1,
                          "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
                          "config": {"workload": res["workload"]}, "eight_layer": res}), flush=True)
        return

    import synth
    import paper_2607_20791_amd as rgd
    from paper_2607_20791_amd import session

    assert torch.cuda.is_available(), "no GPU visible"
    w = synth.LAYER_P8192
    P = w.synthetic_prefix
    Pp = w.prefix_positions
    k, c, N, S = w.probe_k, 3, w.n_branches, w.steps
    t_setup = time.perf_counter()
    log("generating weights ...")
    weights = synth.model_weights(w)
    kp, vp = synth.synthetic_prefix_kv(w, 0)
    last_tok = synth.prompt_tokens(w)[0, 0]
    log(f"weights ready in {time.perf_counter() - t_setup:.1f} s; uploading")
    model = session.build_model(weights, max_rows=N, max_pos=Pp + S + k)
    kv = session.alloc_kv(model, w, max_prompts=1, max_prefix=Pp,
                          n_pages=N * ((S - 1 + 15) // 16) + 4)
    session.fill_prefix(kv, 0, kp, vp)
    dev = "cuda"
    tok = torch.tensor([[int(last_tok)]], dtype=torch.int32, device=dev)
    last = torch.empty(1, w.vocab, dtype=torch.float32, device=dev)
    ptok = torch.empty(1, k, dtype=torch.int32, device=dev)
    plen = torch.empty(1, dtype=torch.int32, device=dev)
    ev = torch.empty(1, dtype=torch.int32, device=dev)
    out = torch.empty(1, N, S, dtype=torch.int32, device=dev)
    seeds = torch.arange(N, dtype=torch.int64, device=dev)

    def prefill():
        kv.set_prefix_len(0, P)
        rgd.prefill_kv(model, kv, tok, P, last)

    if args.table == "typical":
        off, toks = synth.random_table(w)
    else:
        # entry equal to the first 15 greedy tokens, differing at token 16: a
        # full-length miss (greedy tokens from a T=0 run of the same path)
        prefill()
        g = torch.empty(1, 1, k, dtype=torch.int32, device=dev)
        rgd.sample_continuations(model, kv, last, [0], 1, k, 0.0, 0.0, seeds[:1], g)
        gl = g[0, 0].cpu().numpy()
        ent = list(gl[:15]) + [int((gl[15] + 1) % w.vocab)]
        off0, toks0 = synth.random_table(w)
        off = np.concatenate([[0, 16], off0[1:] + 16]).astype(np.int32)
        toks = np.concatenate([ent, toks0]).astype(np.int32)
    table = rgd.Table(off, toks)

    def step(timed=False):
        tp = time.perf_counter()
        prefill()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        rgd.probe(model, kv, last, table, 1, k, c, -1, ptok, plen, ev)
        dec, miss = rgd.gate(kv, ev, 1)
        t1 = time.perf_counter()
        if len(miss):
            if timed:
                rgd.timing_enable(model, TIMING_PERIOD)
            rgd.sample_continuations(model, kv, last, list(miss), N, S, w.temperature, w.min_p,
                                     seeds, out)
            if timed:
                rgd.timing_enable(model, 0)
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        n_probe = int(plen.item())
        return n_probe, len(miss), t1 - t0, t2 - t1, t0 - tp

    # the library creates its timer events on the first enable: do that outside
    # the timed region
    rgd.timing_enable(model, 1)
    rgd.timing_enable(model, 0)
    log("warmup ...")
    for _ in range(args.warmup):
        step()
    rgd.timing_read(model)
    torch.cuda.synchronize()
    log("timed steps ...")
    t_start = time.perf_counter()
    recs = [step(timed=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    rgd.check_status(model)
    tim = rgd.timing_read(model)
    tokens = sum(r[0] + r[1] * N * S for r in recs)
    returned = sum((r[1] * N * S) if r[1] else r[0] for r in recs)
    probe_s = sum(r[2] for r in recs)
    sample_s = sum(r[3] for r in recs)
    prefill_s = sum(r[4] for r in recs)
    # the timed path: probe + gate + sampling, each step bracketed by device
    # synchronisations; the prompt's prefill (its last token over the resident
    # prefix) is excluded from the metric and reported on its own
    path_s = probe_s + sample_s

    lm_b, lm_f, att_b, att_f, samp_b = algorithmic(w, N, Pp, range(1, S))
    n_miss_steps = sum(1 for r in recs if r[1])
    res = {}
    if n_miss_steps:
        lm_ms, lm_n = tim["lm_head"]
        at_ms, at_n = tim["attention"]
        ap_ms, ap_n = tim["attn_prefix"]
        sp_ms, sp_n = tim["sampler"]
        st_ms, st_n = tim["step"]
        lm_avg = lm_ms / lm_n
        lm_gbs = lm_b / (lm_avg * 1e-3) / 1e9
        timed = timed_steps(len(att_b), "attention")  # decode step i+1
        att_total_b = sum(att_b[i] for i in timed) * n_miss_steps
        att_gbs = att_total_b / (at_ms * 1e-3) / 1e9
        attp_total_b = (2 * Pp * w.n_kv_heads * w.head_dim * 2) * ap_n
        attp_gbs = attp_total_b / (ap_ms * 1e-3) / 1e9
        att_tflops = sum(att_f[i] for i in timed) * n_miss_steps / (at_ms * 1e-3) / 1e12
        samp_gbs = samp_b * sp_n / (sp_ms * 1e-3) / 1e9
        res = {
            "roofline": {"bound": "hbm", "kernel": "lm_head_gemm_bf16", "achieved": round(lm_gbs, 1),
                         "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(lm_gbs / HBM_PEAK_GBS, 4),
                         "traffic": measured_traffic(), "avg_us": round(lm_avg * 1e3, 2),
                         "bytes_per_launch": lm_b,
                         "mfma_util": round(lm_f / (lm_avg * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4)},
            "kernels": {
                "attention": {"bound": "hbm", "achieved": round(att_gbs, 1), "peak": HBM_PEAK_GBS,
                              "unit": "GB/s", "frac": round(att_gbs / HBM_PEAK_GBS, 4),
                              "avg_us": round(at_ms / at_n * 1e3, 2), "launches": at_n,
                              "tflops": round(att_tflops, 1),
                              "mfma_frac": round(att_tflops / BF16_PEAK_TFLOPS, 4)},
                "attention_prefix_kernel": {"achieved": round(attp_gbs, 1), "unit": "GB/s",
                                            "frac": round(attp_gbs / HBM_PEAK_GBS, 4),
                                            "avg_us": round(ap_ms / ap_n * 1e3, 2)},
                "sampler": {"bound": "hbm", "achieved": round(samp_gbs, 1), "peak": HBM_PEAK_GBS,
                            "unit": "GB/s", "frac": round(samp_gbs / HBM_PEAK_GBS, 4),
                            "avg_us": round(sp_ms / sp_n * 1e3, 2), "bytes_per_launch": samp_b},
                "decode_step": {"avg_us": round(st_ms / st_n * 1e3, 2), "launches": st_n},
            },
        }
    line = {
        "metric": METRIC, "value": round(tokens / path_s, 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(path_s / args.steps * 1e3, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "prefix_positions": Pp, "branches": N, "steps": S,
                   "probe_k": k, "check_cadence": c, "temperature": w.temperature,
                   "min_p": w.min_p, "table": args.table, "page_size": 16},
        "tokens_decoded": tokens, "tokens_returned": returned,
        "gate_overhead": round(probe_s / sample_s, 5) if sample_s > 0 else None,
        "probe_gate_ms_per_step": round(probe_s / args.steps * 1e3, 3),
        "sampling_ms_per_step": round(sample_s / args.steps * 1e3, 3),
        "prefill_ms_per_step": round(prefill_s / args.steps * 1e3, 3),
        "wall_ms_per_step_with_prefill": round(elapsed / args.steps * 1e3, 3),
    }
    line.update(res)
    log("p-less sampling ...")
    line["pless"] = pless_variant(rgd, torch, model, kv, w, last, N, S, seeds, out, sample_s / args.steps * 1e3)
    log("gate variants ...")
    line["gate_variants"] = gate_variants(rgd, torch, model, kv, w, last, last_tok, table, prefill, k, c,
                                          sample_s / args.steps * 1e3)
    # the gate-overhead target is judged on the full-length miss (a probe that
    # decodes all k tokens before it fails); the typical miss fails at token 1
    line["gate_overhead_full_length_miss"] = line["gate_variants"]["hard_adversarial"]["overhead"]
    log("sampler sweep ...")
    line["sampler_sweep"] = sampler_sweep(rgd, torch)
    if not args.no_eight_layer:
        # the end-to-end workload (8 layers, 32 prompts of 1024 tokens, gated
        # against ungated) on its own model, after this one is released
        del model, kv
        torch.cuda.empty_cache()
        log("8-layer gated vs ungated ...")
        line["eight_layer"] = eight_layer(rgd, torch, reps=1)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle ...")
        line["cpu_baseline"] = cpu_baseline(weights, w, P, last_tok, kp, vp)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
