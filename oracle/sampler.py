"""Token selection: greedy argmax and temperature-scaled min-p sampling.

Section 3 defines S_{T,theta}(M, p) as ordinary high-temperature sampling with a
truncation rule; Section 1 names min-p as a truncation method for the high
temperature regime.  The reading used throughout (temperature first, then the
min-p mask, then one inverse-CDF draw in ascending token-id order) is:

    m   = max_i z_i
    w_i = exp((z_i - m) / T)              (= p_i / p_max of softmax(z / T))
    keep i  iff  w_i >= p_min              (i.e. p_i >= p_min * p_max)
    W   = sum of kept w_i
    C_i = running sum of kept w_j, j <= i
    return the smallest kept i with C_i > u * W

T = 0 is greedy decoding: the first index of the maximum logit.
All arithmetic is float64 on the given logits.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np


def argmax(z) -> int:
    """Greedy token: first index attaining the maximum (ties -> lowest id)."""
    return int(np.argmax(np.asarray(z)))


def logit_margin_argmax(z) -> float:
    """Gap between the largest and second-largest logit (0 on a tie)."""
    z = np.asarray(z, dtype=np.float64)
    if z.size < 2:
        return math.inf
    top2 = np.partition(z, -2)[-2:]
    return float(top2[1] - top2[0])


def minp_weights(z, T: float, p_min: float):
    """Returns (w, kept): w_i = exp((z_i - max z)/T) and the min-p mask."""
    z = np.asarray(z, dtype=np.float64)
    m = z.max()
    w = np.exp((z - m) / T)
    return w, w >= p_min


@dataclass
class Draw:
    token: int
    logit_margin: float   # min_i |(z_i - m)/T - ln p_min|  (mask decisions)
    cdf_margin: float     # distance of u*W to the nearest CDF edge, over W


def sample_minp(z, T: float, p_min: float, u: float) -> Draw:
    """One min-p draw with uniform u in [0, 1).  T == 0 gives argmax."""
    z = np.asarray(z, dtype=np.float64)
    if T == 0.0:
        return Draw(argmax(z), logit_margin_argmax(z), math.inf)
    w, kept = minp_weights(z, T, p_min)
    wk = np.where(kept, w, 0.0)
    total = wk.sum()
    cdf = np.cumsum(wk)
    t = u * total
    kept_idx = np.flatnonzero(kept)
    above = kept_idx[cdf[kept_idx] > t]
    tok = int(above[0]) if above.size else int(kept_idx[-1])
    edges = np.concatenate(([0.0], cdf[kept_idx]))
    cdf_margin = float(np.min(np.abs(edges - t)) / total)
    lmarg = float(np.min(np.abs((z - z.max()) / T - math.log(p_min)))) if p_min > 0 else math.inf
    return Draw(tok, lmarg, cdf_margin)


def kept_probabilities(z, T: float, p_min: float) -> np.ndarray:
    """The distribution a min-p draw follows: kept w_i renormalised."""
    w, kept = minp_weights(z, T, p_min)
    wk = np.where(kept, w, 0.0)
    return wk / wk.sum()


def sample_minp_many(z, T: float, p_min: float, us) -> list:
    """sample_minp for many uniforms on one row (same definition; the kept
    weights and running sums are formed once)."""
    z = np.asarray(z, dtype=np.float64)
    w, kept = minp_weights(z, T, p_min)
    wk = np.where(kept, w, 0.0)
    total = wk.sum()
    cdf = np.cumsum(wk)
    kept_idx = np.flatnonzero(kept)
    ck = cdf[kept_idx]
    edges = np.concatenate(([0.0], ck))
    lmarg = float(np.min(np.abs((z - z.max()) / T - math.log(p_min)))) if p_min > 0 else math.inf
    out = []
    for u in np.asarray(us, dtype=np.float64):
        t = u * total
        j = int(np.searchsorted(ck, t, side="right"))      # first kept running sum > t
        tok = int(kept_idx[min(j, kept_idx.size - 1)])
        k = int(np.searchsorted(edges, t))
        near = edges[max(k - 1, 0):k + 1]
        out.append(Draw(tok, lmarg, float(np.min(np.abs(near - t)) / total)))
    return out
