"""Residual-stream classifier pre-check (Appendix A) and the adaptive gate.

A logistic readout of the last prompt token's residual stream after a chosen
layer, P = 1 / (1 + exp(-(w . h + b))) with d + 1 parameters, predicts whether
the greedy answer would start as a refusal.  A prompt with P <= theta skips the
greedy check (zero check tokens) and is sampled directly; any other prompt goes
through the refusal gate of Algorithm 1 (here the hard gate, or the soft gate
of Appendix C).  The paper's trained classifiers are not available: tests and
timing use random weights, so only the computation and the decision rule are
reproduced, not the classifier's accuracy.

Test infrastructure only (the oracle); the HIP path shares no code with it.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import gate, rgd


def residual_score(h, w, b: float) -> float:
    """P = sigmoid(w . h + b) in float64."""
    z = float(np.dot(np.asarray(w, np.float64), np.asarray(h, np.float64))) + float(b)
    return 1.0 / (1.0 + np.exp(-z))


@dataclass
class AdaptiveResult:
    score: float
    skipped: bool
    gated: rgd.GatedResult


def adaptive_gated(model, prompt, table, k: int, seeds, steps: int, T: float, p_min: float,
                   layer: int, w, b: float, theta: float, soft=None, eos: int = -1,
                   min_match: int = 2) -> AdaptiveResult:
    """Prefill once; score the last prompt token's residual after `layer`; a
    score <= theta samples directly, otherwise the gate decides (soft: (c, K,
    rho) for the soft gate of Appendix C, None for the hard gate)."""
    from .model import KVCache
    prefix = KVCache(model.cfg.n_layers)
    taps = {}
    last = model.prefill(prompt, prefix, taps=taps)
    p = residual_score(taps[layer], w, b)
    if p <= theta:
        br = [rgd.sample_branch(model, prefix, last, int(s), steps, T, p_min) for s in seeds]
        return AdaptiveResult(p, True, rgd.GatedResult(False, [], gate.INCOMPAT, br))
    if soft is None:
        g = rgd.refusal_gated(model, prompt, table, k, seeds, steps, T, p_min, eos, min_match,
                              prefix=prefix, last_logits=last)
    else:
        c, K, rho = soft
        q, ev = rgd.soft_greedy_probe(model, prefix, last, table, k, c, K, rho, eos, min_match)
        if gate.is_hit(ev):
            g = rgd.GatedResult(True, q, ev, [])
        else:
            br = [rgd.sample_branch(model, prefix, last, int(s), steps, T, p_min) for s in seeds]
            g = rgd.GatedResult(False, q, ev, br)
    return AdaptiveResult(p, False, g)
