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
"""
from __future__ import annotations

INCOMPAT, STOP, MAXLEN = 0, 1, 2


def is_prefix(a, b) -> bool:
    """True iff sequence a is a prefix of sequence b."""
    return len(a) <= len(b) and list(b[:len(a)]) == list(a)


def compatible(q, table, min_match: int = 2) -> bool:
    """C(q, P) on token ids: q is a prefix of an entry, or an entry is a prefix
    of q; entries shorter than min_match are ignored."""
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


def is_hit(event: int) -> bool:
    """Gate decision: the greedy probe is returned on STOP or MAXLEN."""
    return event in (STOP, MAXLEN)
