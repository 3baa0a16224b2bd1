"""Algorithm 1 end to end on the oracle decoder (Section 3).

A prompt is prefilled once; its KV cache is shared by the probe and by every
sampled branch (the probe's own positions are discarded on a miss, and each
branch restarts from the prompt, so branch positions start right after the
prompt).  A hit returns the greedy probe; a miss returns N independent min-p
draws sequences, branch b using Philox key seeds[b] and counter (step, 0).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import gate, philox, pless, sampler
from .model import Decoder, KVCache


@dataclass
class BranchResult:
    tokens: list
    draws: list        # sampler.Draw per step (margins for reporting)
    logits: list       # per-step logits (only when keep_logits)


def sample_branch(model: Decoder, prefix: KVCache, last_logits, seed: int, steps: int,
                  T: float, p_min: float, forced=None, keep_logits: bool = False,
                  stream: int = 0, truncation: str = "minp") -> BranchResult:
    """S_{T,theta}(M, p) for one branch: token s uses Philox counter (s, stream).
    With `forced`, token forced[s] (not the drawn one) is fed after step s.
    truncation "minp" (threshold p_min) or "pless" (p_min unused)."""
    tail = KVCache(model.cfg.n_layers)
    logits = np.asarray(last_logits, np.float64)
    toks, draws, kept = [], [], []
    for s in range(steps):
        if keep_logits:
            kept.append(logits)
        u = float(philox.uniform(seed, s, stream))
        d = pless.sample_pless(logits, T, u) if truncation == "pless" else sampler.sample_minp(logits, T, p_min, u)
        toks.append(d.token)
        draws.append(d)
        if s + 1 < steps:
            feed = int(forced[s]) if forced is not None else d.token
            logits = model.decode(feed, prefix, tail)
    return BranchResult(toks, draws, kept)


def greedy_probe(model: Decoder, prefix: KVCache, last_logits, table, k: int, eos: int = -1,
                 min_match: int = 2):
    """The probe of Algorithm 1 against the shared prompt cache."""
    tail = KVCache(model.cfg.n_layers)

    def nxt(q):
        return model.decode(q[-1], prefix, tail)

    return gate.probe(last_logits, nxt, table, k, eos, min_match)


def fixed_greedy_probe(model: Decoder, prefix: KVCache, last_logits, table, k: int, eos: int = -1,
                       min_match: int = 2):
    """The probe with no compatibility gate (greedy decoding to k tokens, the
    detector applied once at the end) against the shared prompt cache: the
    fixed-probe ablation (Appendix B) and the naive greedy answer (Section 3)."""
    tail = KVCache(model.cfg.n_layers)

    def nxt(q):
        return model.decode(q[-1], prefix, tail)

    return gate.fixed_probe(last_logits, nxt, table, k, eos, min_match)


def soft_greedy_probe(model: Decoder, prefix: KVCache, last_logits, table, k: int, c: int, K: int,
                      rho: float, eos: int = -1, min_match: int = 2, steps: list | None = None):
    """The probe of the soft compatibility-gate variant (Appendix C) against the
    shared prompt cache."""
    tail = KVCache(model.cfg.n_layers)

    def nxt(q):
        return model.decode(q[-1], prefix, tail)

    return gate.soft_probe(last_logits, nxt, table, k, c, K, rho, eos, min_match, steps)


@dataclass
class GatedResult:
    hit: bool
    probe: list
    event: int
    branches: list     # BranchResult per branch on a miss


def refusal_gated(model: Decoder, prompt, table, k: int, seeds, steps: int, T: float,
                  p_min: float, eos: int = -1, min_match: int = 2,
                  prefix: KVCache | None = None, last_logits=None) -> GatedResult:
    if prefix is None:
        prefix = KVCache(model.cfg.n_layers)
        last_logits = model.prefill(prompt, prefix)
    q, ev = greedy_probe(model, prefix, last_logits, table, k, eos, min_match)
    if gate.is_hit(ev):
        return GatedResult(True, q, ev, [])
    br = [sample_branch(model, prefix, last_logits, int(s), steps, T, p_min) for s in seeds]
    return GatedResult(False, q, ev, br)
