"""p-less truncation for the sampled continuations.

The experiments of Section 4 sample every high-temperature continuation with
p-less sampling (Tan et al.), which the paper cites without stating its rule.
The rule taken here is the one of the p-less paper: a token is kept when its
probability is at least the probability that two independent draws from the
distribution agree, sum_j p_j^2.  It has no parameter.  As for min-p,
temperature comes first:

    p   = softmax(z / T)                   (float64)
    thr = sum_j p_j^2
    keep i  iff  p_i >= thr
    W   = sum of kept p_i
    C_i = running sum of kept p_j over j <= i (ascending token id)
    return the smallest kept i with C_i > u * W

The most probable token is always kept: sum_j p_j^2 <= p_max * sum_j p_j =
p_max.  T = 0 is greedy decoding (argmax).

Parity status: the rule itself comes from the cited p-less paper, not from
this paper, so this module pins the computation (closed forms, brute force,
invariants, draw statistics), not the choice of rule.

Test infrastructure only (the oracle); the HIP path shares no code with it.
"""
from __future__ import annotations

import math

import numpy as np

from .sampler import Draw, argmax, logit_margin_argmax


def pless_probabilities(z, T: float):
    """Returns (p, thr, kept): p = softmax(z / T), thr = sum p^2, kept = p >= thr."""
    z = np.asarray(z, dtype=np.float64)
    e = np.exp((z - z.max()) / T)
    p = e / e.sum()
    thr = float(np.sum(p * p))
    return p, thr, p >= thr


def _membership_margin(p, thr) -> float:
    """min_i |ln p_i - ln thr| over tokens with p_i > 0 (mask decisions near the edge)."""
    pos = p[p > 0]
    return float(np.min(np.abs(np.log(pos) - math.log(thr))))


def sample_pless(z, T: float, u: float) -> Draw:
    """One p-less draw with uniform u in [0, 1).  T == 0 gives argmax."""
    z = np.asarray(z, dtype=np.float64)
    if T == 0.0:
        return Draw(argmax(z), logit_margin_argmax(z), math.inf)
    p, thr, kept = pless_probabilities(z, T)
    pk = np.where(kept, p, 0.0)
    total = pk.sum()
    cdf = np.cumsum(pk)
    t = u * total
    kept_idx = np.flatnonzero(kept)
    above = kept_idx[cdf[kept_idx] > t]
    tok = int(above[0]) if above.size else int(kept_idx[-1])
    edges = np.concatenate(([0.0], cdf[kept_idx]))
    return Draw(tok, _membership_margin(p, thr), float(np.min(np.abs(edges - t)) / total))


def kept_probabilities(z, T: float) -> np.ndarray:
    """The distribution a p-less draw follows: kept p_i renormalised."""
    p, _, kept = pless_probabilities(z, T)
    pk = np.where(kept, p, 0.0)
    return pk / pk.sum()


def sample_pless_many(z, T: float, us) -> list:
    """sample_pless for many uniforms on one row (kept set and running sums
    formed once)."""
    z = np.asarray(z, dtype=np.float64)
    p, thr, kept = pless_probabilities(z, T)
    pk = np.where(kept, p, 0.0)
    total = pk.sum()
    cdf = np.cumsum(pk)
    kept_idx = np.flatnonzero(kept)
    ck = cdf[kept_idx]
    edges = np.concatenate(([0.0], ck))
    lmarg = _membership_margin(p, thr)
    out = []
    for u in np.asarray(us, dtype=np.float64):
        t = u * total
        j = int(np.searchsorted(ck, t, side="right"))
        tok = int(kept_idx[min(j, kept_idx.size - 1)])
        k = int(np.searchsorted(edges, t))
        near = edges[max(k - 1, 0):k + 1]
        out.append(Draw(tok, lmarg, float(np.min(np.abs(near - t)) / total)))
    return out
