"""Refusal-prefix compatibility, the greedy probe and the gate (Section 3,
Algorithm 1; Appendix D for the token-level matching rule).

Compatibility C(q, P) holds when the probe q is a prefix of some refusal
prefix pi in P, or some pi is a prefix of q.  The runtime detector matches
token prefixes with a two-token minimum (Appendix D); the reading used here is
that table entries shorter than `min_match` tokens never match.  The workloads
have no tokenizer, so the predicate is applied to token ids directly.

Probe: the first token is the argmax of the prompt's last-position logits; each
further token is the argmax after feeding the probe so far.  After each token:
if q is incompatible the probe ends with INCOMPAT (the prompt is sampled);
otherwise a stop token ends it with STOP and reaching k tokens with MAXLEN
(both return the greedy probe).  Algorithm 1 splits the loop into a c-token
gate and a post-cap probe B_M with the same three events; the decision does not
depend on c.

Soft variant (Appendix C): during the first c tokens, a greedy token that would
make q incompatible is not final.  Among the K most probable next tokens, those
that keep q compatible carry a probability mass m; if that set is not empty and
m >= rho, its most probable token is appended instead and the probe goes on.
After c tokens the hard rule applies (the post-cap probe B_M).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

INCOMPAT, STOP, MAXLEN = 0, 1, 2


def is_prefix(a, b) -> bool:
    """True iff sequence a is a prefix of sequence b."""
    return len(a) <= len(b) and list(b[:len(a)]) == list(a)


def compatible(q, table, min_match: int = 2) -> bool:
    """C(q, P) on token ids: q is a prefix of an entry, or an entry is a prefix
    of q; entries shorter than min_match are ignored.  table None: no refusal
    set at all, the fixed-length probe of the ablations (every q passes)."""
    if table is None:
        return True
    q = [int(t) for t in q]
    for e in table:
        e = [int(t) for t in e]
        if len(e) < min_match:
            continue
        if is_prefix(q, e) or is_prefix(e, q):
            return True
    return False


def table_entries(offsets, tokens):
    """CSR (offsets[n+1], tokens) -> list of token lists."""
    return [list(tokens[offsets[i]:offsets[i + 1]]) for i in range(len(offsets) - 1)]


def probe(first_logits, next_logits, table, k: int, eos: int = -1, min_match: int = 2,
          pick=None):
    """Greedy probe of at most k tokens.  next_logits(q) returns the logits after
    feeding the whole probe q (its last token is the new input).  pick(logits)
    chooses the greedy token (default: oracle argmax).  Returns (q, event)."""
    if pick is None:
        from .sampler import argmax as pick
    q = []
    logits = first_logits
    while True:
        y = pick(logits)
        q.append(int(y))
        if not compatible(q, table, min_match):
            return q, INCOMPAT
        if eos >= 0 and y == eos:
            return q, STOP
        if len(q) >= k:
            return q, MAXLEN
        logits = next_logits(q)


def fixed_probe(first_logits, next_logits, table, k: int, eos: int = -1, min_match: int = 2,
                pick=None):
    """Probe without the compatibility gate: greedy decoding runs to k tokens
    (or to a stop token) whatever the tokens are, and the refusal detector is
    applied once to the finished probe.  This is the fixed-probe ablation of
    Appendix B (k = 32) and, with k equal to the full response budget L, the
    naive greedy-then-high-temperature approach of Section 3 (a complete
    greedy answer first, sampling only when it is not a refusal).  Returns
    (q, event): INCOMPAT when C(q) fails (the prompt is sampled), otherwise
    STOP if decoding ended on the stop token and MAXLEN if it reached k."""
    if pick is None:
        from .sampler import argmax as pick
    q = []
    logits = first_logits
    while True:
        y = int(pick(logits))
        q.append(y)
        if (eos >= 0 and y == eos) or len(q) >= k:
            break
        logits = next_logits(q)
    if not compatible(q, table, min_match):
        return q, INCOMPAT
    return q, (STOP if eos >= 0 and q[-1] == eos else MAXLEN)


def top_k(z, K: int):
    """The K most probable tokens of logits z, most probable first (equal logits:
    lower id first), with their probabilities under softmax(z) over the whole
    vocabulary (temperature 1: the model's own next-token distribution)."""
    z = np.asarray(z, np.float64)
    order = np.lexsort((np.arange(len(z)), -z))
    w = np.exp(z - z.max())
    p = w / w.sum()
    return [(int(i), float(p[i])) for i in order[:K]]


@dataclass
class SoftStep:
    """What a soft step decided, with the margins that make it fragile under
    rounding: the gap between the K-th and (K+1)-th logit (top-K membership) and
    the relative distance |m - rho| / max(m, rho) of the mass test; None where
    the step did not use them."""
    greedy: int
    appended: int
    mass: float | None = None
    topk_gap: float | None = None
    rho_margin: float | None = None


def soft_step(q, logits, table, c: int, K: int, rho: float, min_match: int = 2):
    """One probe step from probe q with next-token logits: returns (token,
    passed, SoftStep or None).  The greedy token is taken when q stays
    compatible; otherwise, while len(q) < c (tokens 1..c are soft steps), the
    most probable compatible token of the top K is taken when the compatible
    ones of the top K carry mass >= rho.  passed False: the greedy token failed
    (INCOMPAT).  The SoftStep is returned for soft steps that met an
    incompatible greedy token."""
    from .sampler import argmax
    q = list(q)
    y = int(argmax(logits))
    if compatible(q + [y], table, min_match):
        return y, True, None
    if len(q) >= c:
        return y, False, None
    cand = top_k(logits, K)
    alts = [(a, pa) for a, pa in cand if compatible(q + [a], table, min_match)]
    mass = sum(pa for _, pa in alts)
    zs = np.sort(np.asarray(logits, np.float64))[::-1]
    gap = float(zs[K - 1] - zs[K]) if K < len(zs) else None
    ok = bool(alts) and mass >= rho
    scale = max(mass, abs(rho))
    info = SoftStep(y, alts[0][0] if ok else y, mass, gap, abs(mass - rho) / scale if scale > 0 else 0.0)
    return (alts[0][0], True, info) if ok else (y, False, info)


def soft_probe(first_logits, next_logits, table, k: int, c: int, K: int, rho: float,
               eos: int = -1, min_match: int = 2, steps: list | None = None):
    """Probe with the soft compatibility gate (Appendix C, Algorithm 2): tokens
    1..c are soft steps, later ones follow the hard rule.  Returns (q, event);
    on INCOMPAT the last token of q is the greedy token that failed.  `steps`,
    when given, collects one SoftStep per soft step that met an incompatible
    greedy token."""
    q = []
    logits = first_logits
    while True:
        t, passed, info = soft_step(q, logits, table, c, K, rho, min_match)
        if info is not None and steps is not None:
            steps.append(info)
        q.append(t)
        if not passed:
            return q, INCOMPAT
        if eos >= 0 and t == eos:
            return q, STOP
        if len(q) >= k:
            return q, MAXLEN
        logits = next_logits(q)


def is_hit(event: int) -> bool:
    """Gate decision: the greedy probe is returned on STOP or MAXLEN."""
    return event in (STOP, MAXLEN)
